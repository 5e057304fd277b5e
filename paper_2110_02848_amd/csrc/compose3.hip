// Kernels of the simultaneous composition of three transducers, C = A o B o
// D (the N-way composition the paper names as the next step after its
// two-input one, Section 5), for gfx950.
//
// A state of C is a key (qa, qb, f1, qd, f2).  (qa, qb, f1) is a state of
// T = A o B, read on the fly: its arcs are the two-input moves (a matching
// pair of arcs of A and B; an A arc with output epsilon, only when f1 = 0;
// a B arc with input epsilon, setting f1 = epsOutA(qa)).  The key composes
// T with D by the same three rules with filter bit f2: a T-arc whose output
// z is not epsilon with a D arc of input z; a T-arc with output epsilon
// alone, only when f2 = 0; a D arc with input epsilon alone, setting f2 =
// epsOutT(qa, qb, f1) (whether that T-state has an arc with output
// epsilon).  Weights: a T-match is w(a) + w(b), a match with D adds w(d)
// after it; single arcs copy their weight.
//
// The key space is the product of three state sets, far too large for a
// bitmap, so keys are 64-bit, packed so that numeric order is (qa, qb, f1,
// qd, f2) order, and deduplicated in an open-addressing hash set whose slot
// index names the state during the search.
//
// Work units of a key, in canonical order: its A arcs with output epsilon
// (only when f1 = f2 = 0), its B arcs with input epsilon, its D arcs with
// input epsilon, then one unit per non-epsilon arc of whichever of A and B
// has fewer: the unit of the first arc of a label joins the label's arcs
// of A (outer, by arc index) with those of B (inner), each T-arc with the D
// bucket of its output; later arcs of the same label do nothing.  So the
// moves come out in canonical (l, a, b, d) order (l the label A and B were
// matched on, 0 for the epsilon units; a missing arc last) and a key whose
// B state has one arc (a lexicon word) has one unit however many arcs its
// A state has.
//
// The search goes level by level.  A thread takes a frontier key (or a
// chunk of CHUNK3 units of a key with more than WALK3), expands it and goes
// on depth-first
// with the first new key it reached (up to CHAIN3 keys), so a word of a
// lexicon is one thread's walk; other new keys join the next frontier, and
// heavy keys met on a walk are cut into chunks.  Every generated arc
// (source slot, target slot) is appended to an arc list, and new keys to
// the next frontier, one atomic per wavefront.  Keys with one move along a
// chain of B (a word's letters) are crossed by a chain jump that inserts
// the keys it reaches together, and a lexicon root's chunk of word entries
// is expanded in one batch (see jump3 and expand_beps).
// Co-accessibility runs backwards over that arc list (in-arcs grouped by a
// radix sort of the arcs by target, their run boundaries and a scan); the
// keys of a jump's chain segment are claimed together.  The trim keys are sorted (radix sort of
// the 64-bit keys): a state's id is its rank.  Count and fill give a state
// with at most LIGHT3 units one thread and a heavier one a workgroup (its
// threads take its units in turn); per-unit counts are scanned into every
// unit's first arc position.
#include "internal.h"

namespace fstc {

namespace {

typedef unsigned long long ull;

constexpr ull EMPTY3 = ~0ull;
constexpr uint32_t NO_SLOT = 0xFFFFFFFFu;
constexpr uint32_t LIGHT3 = 8;    // output: units of a state one thread writes
constexpr uint32_t WALK3 = 8;     // search: units of a key a walk expands in place
constexpr int PROBE_MAX = 256;    // hash probes before the table counts as full
constexpr uint32_t BF_EPS_EPS = 1u, BF_EPS_OUT = 2u;  // B state flags

unsigned grid3(size_t n, unsigned cap = 4096) {
  size_t g = (n + NT - 1) / NT;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

// The state id in an arc record's neighbour field.
__device__ __forceinline__ uint32_t nbr_of_arc(int32_t y) { return (uint32_t)(y & NBR_MASK); }

__device__ __forceinline__ ull mix64(ull x) {
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

__device__ __forceinline__ ull pack3(const Problem3 &P, uint32_t qa, uint32_t qb, uint32_t f1,
                                     uint32_t qd, uint32_t f2) {
  return (((((ull)qa << P.shB | qb) << 1 | f1) << P.shD | qd) << 1) | f2;
}

struct Key3 {
  uint32_t qa, qb, f1, qd, f2;
};

__device__ __forceinline__ Key3 unpack3(const Problem3 &P, ull k) {
  Key3 s;
  s.f2 = (uint32_t)(k & 1ull);
  k >>= 1;
  s.qd = (uint32_t)(k & ((1ull << P.shD) - 1ull));
  k >>= P.shD;
  s.f1 = (uint32_t)(k & 1ull);
  k >>= 1;
  s.qb = (uint32_t)(k & ((1ull << P.shB) - 1ull));
  s.qa = (uint32_t)(k >> P.shB);
  return s;
}

// The set is probed in aligned groups of four slots (32 bytes, one cache
// line sector), group after group from the key's hash: a key sits in the
// first group of its sequence with a free slot when it was inserted.
constexpr uint32_t HGROUP = 4;

__device__ __forceinline__ void load_group(const Problem3 &P, uint32_t h, ull g[HGROUP]) {
  const ulonglong2 *q = reinterpret_cast<const ulonglong2 *>(P.tab + h);
  const ulonglong2 a = q[0], b = q[1];
  g[0] = a.x;
  g[1] = a.y;
  g[2] = b.x;
  g[3] = b.y;
}

// Slot of key k: inserted if absent (fresh), NO_SLOT (and the overflow
// flag) if PROBE_MAX slots in a row are taken.  Plain loads first: a slot
// never changes once set, so a stale EMPTY only sends the thread to the CAS.
__device__ __forceinline__ uint32_t h_insert(const Problem3 &P, ull k, bool &fresh,
                                             uint32_t *overflow) {
  uint32_t h = (uint32_t)mix64(k) & P.hmask & ~(HGROUP - 1u);
  fresh = false;
  for (int p = 0; p < PROBE_MAX; p += HGROUP) {
    ull g[HGROUP];
    load_group(P, h, g);
#pragma unroll
    for (uint32_t j = 0; j < HGROUP; ++j)
      if (g[j] == k) return h + j;
#pragma unroll
    for (uint32_t j = 0; j < HGROUP; ++j) {
      if (g[j] != EMPTY3) continue;
      const ull old = atomicCAS(P.tab + h + j, EMPTY3, k);
      if (old == EMPTY3) {
        fresh = true;
        return h + j;
      }
      if (old == k) return h + j;
    }
    h = (h + HGROUP) & P.hmask;
  }
  atomicOr(overflow, 1u);
  return NO_SLOT;
}

// Slot of key k, or NO_SLOT if it is not in the set.
__device__ __forceinline__ uint32_t h_find(const Problem3 &P, ull k) {
  uint32_t h = (uint32_t)mix64(k) & P.hmask & ~(HGROUP - 1u);
  for (int p = 0; p < PROBE_MAX; p += HGROUP) {
    ull g[HGROUP];
    load_group(P, h, g);
    bool empty = false;
#pragma unroll
    for (uint32_t j = 0; j < HGROUP; ++j) {
      if (g[j] == k) return h + j;
      empty = empty || g[j] == EMPTY3;
    }
    if (empty) return NO_SLOT;
    h = (h + HGROUP) & P.hmask;
  }
  return NO_SLOT;
}

// Append x for every lane with `want`, one atomic per wavefront; false (and
// the overflow flag) past the capacity.
template <class T>
__device__ __forceinline__ void wave_append(bool want, T x, T *list, ull cap, uint32_t *count,
                                            uint32_t *overflow) {
  const ull m = __ballot(want);
  if (m == 0) return;
  const int leader = __ffsll(m) - 1;
  uint32_t base = 0;
  if ((int)__lane_id() == leader) base = atomicAdd(count, (uint32_t)__popcll(m));
  base = __shfl(base, leader, WAVE);
  if (want) {
    const ull pos = (ull)base + (ull)__popcll(m & __lanemask_lt());
    if (pos < cap) list[pos] = x;
    else atomicOr(overflow, 1u);
  }
}

// A state's arc group in a label-sorted view: [begin, end), the first
// `neps` arcs with label epsilon.
struct Grp {
  int32_t begin, neps, end, flags;
};
__device__ __forceinline__ Grp grp_of(const View &v, uint32_t q) {
  const int4 r = v.srec[2 * (size_t)q];
  return Grp{r.x, r.y, r.z, r.w};
}

// [lo, hi) of label lab among the non-epsilon arcs [lo, hi) of group q:
// one load from the view's bucket table when it has one, else a binary
// search.
__device__ __forceinline__ void bucket(const View &v, uint32_t q, int32_t lo, int32_t hi,
                                       int32_t lab, int32_t &r0, int32_t &r1) {
  if (v.lut) {
    if ((uint32_t)lab < (uint32_t)v.lstride) {
      const int4 b = v.lut[(size_t)q * (uint32_t)v.lstride + (uint32_t)lab];
      r0 = b.x;
      r1 = b.y;
    } else {
      r0 = r1 = hi;
    }
    return;
  }
  int32_t a = lo, b = hi;
  while (a < b) {
    const int32_t mid = a + ((b - a) >> 1);
    if (v.arec[mid].x < lab) a = mid + 1; else b = mid;
  }
  r0 = a;
  b = hi;
  while (a < b) {
    const int32_t mid = a + ((b - a) >> 1);
    if (v.arec[mid].x <= lab) a = mid + 1; else b = mid;
  }
  r1 = a;
}

// epsOutT(qa, qb, f1): some T-arc out of (qa, qb, f1) has output epsilon.
__device__ __forceinline__ uint32_t eps_out_t(const Problem3 &P, uint32_t qa, uint32_t qb,
                                              uint32_t f1) {
  const Grp ga = grp_of(P.aOut, qa);
  if (f1 == 0 && ga.neps > 0) return 1u;
  const uint32_t bf = P.bflags[qb];
  if (bf & BF_EPS_EPS) return 1u;
  if (!(bf & BF_EPS_OUT)) return 0u;
  // a B arc with input y != eps and output eps, and an A arc with output y
  const Grp gb = grp_of(P.bOut, qb);
  for (int32_t p = gb.begin + gb.neps; p < gb.end; ++p) {
    if (P.bOut.olab[p] != 0) continue;
    int32_t r0, r1;
    bucket(P.aOut, qa, ga.begin + ga.neps, ga.end, P.bOut.arec[p].x, r0, r1);
    if (r0 < r1) return 1u;
  }
  return 0u;
}

// The work units of a key (see the file comment).
struct Units3 {
  Key3 k;
  Grp ga, gb, gd;
  uint32_t nae;      // A-epsilon units (0 unless f1 = f2 = 0)
  uint32_t nm;       // matching units: non-epsilon arcs of the smaller side
  bool joinA;        // the matching units walk A's arcs (else B's)
};
__device__ __forceinline__ Units3 units_of(const Problem3 &P, ull key) {
  Units3 u;
  u.k = unpack3(P, key);
  u.ga = grp_of(P.aOut, u.k.qa);
  u.gb = grp_of(P.bOut, u.k.qb);
  u.gd = grp_of(P.dOut, u.k.qd);
  u.nae = (u.k.f1 == 0 && u.k.f2 == 0) ? (uint32_t)u.ga.neps : 0u;
  const uint32_t na = (uint32_t)(u.ga.end - u.ga.begin - u.ga.neps);
  const uint32_t nb = (uint32_t)(u.gb.end - u.gb.begin - u.gb.neps);
  u.joinA = na <= nb;
  u.nm = (na && nb) ? (u.joinA ? na : nb) : 0u;
  return u;
}
__device__ __forceinline__ uint32_t nunits(const Units3 &u) {
  return u.nae + (uint32_t)u.gb.neps + (uint32_t)u.gd.neps + u.nm;
}

// A T-arc (B's arc at position p of its view, A's arc id ea or -1, target
// (ta, tb, tf1), input label il, weight wt) composed with D: alone when
// its output is epsilon (f2 = 0 only), else with the D bucket of its output.
template <class F>
__device__ __forceinline__ void t_with_d(const Problem3 &P, const Units3 &u, int32_t p, int32_t ea,
                                         uint32_t ta, uint32_t tf1, int32_t il, float wt, F &&f) {
  const int32_t eb = P.bOut.perm[p], z = P.bOut.olab[p];
  const uint32_t tb = nbr_of_arc(P.bOut.arec[p].y);
  if (z == 0) {
    if (u.k.f2 == 0) f(pack3(P, ta, tb, tf1, u.k.qd, 0), il, 0, wt, ea, eb, -1);
    return;
  }
  int32_t d0, d1;
  bucket(P.dOut, u.k.qd, u.gd.begin + u.gd.neps, u.gd.end, z, d0, d1);
  for (int32_t r = d0; r < d1; ++r)
    f(pack3(P, ta, tb, tf1, nbr_of_arc(P.dOut.arec[r].y), 0), il, P.dOut.olab[r],
      wt + P.dOut.w[r], ea, eb, P.dOut.perm[r]);
}

// Calls f(target key, ilabel, olabel, weight, a, b, d) for every move of
// unit j of a key, in canonical order (arc ids; -1 = none).
template <class F>
__device__ __forceinline__ void for_unit3(const Problem3 &P, const Units3 &u, uint32_t j, F &&f) {
  const Key3 &k = u.k;
  if (j < u.nae) {
    // A alone (output epsilon; f1 = f2 = 0): T-arc alone as well
    const int32_t p = u.ga.begin + (int32_t)j;
    f(pack3(P, nbr_of_arc(P.aOut.arec[p].y), k.qb, 0, k.qd, 0), P.aOut.olab[p], 0,
      P.aOut.w[p], P.aOut.perm[p], -1, -1);
    return;
  }
  j -= u.nae;
  if (j < (uint32_t)u.gb.neps) {
    // B alone (input epsilon): T-state (qa, dst b, epsOutA(qa))
    const int32_t p = u.gb.begin + (int32_t)j;
    t_with_d(P, u, p, -1, k.qa, u.ga.neps > 0 ? 1u : 0u, 0, P.bOut.w[p], f);
    return;
  }
  j -= (uint32_t)u.gb.neps;
  if (j < (uint32_t)u.gd.neps) {
    // D alone (input epsilon): f2 = epsOutT of the key's T-state
    const int32_t r = u.gd.begin + (int32_t)j;
    const uint32_t nf2 = eps_out_t(P, k.qa, k.qb, k.f1);
    f(pack3(P, k.qa, k.qb, k.f1, nbr_of_arc(P.dOut.arec[r].y), nf2), 0, P.dOut.olab[r],
      P.dOut.w[r], -1, -1, P.dOut.perm[r]);
    return;
  }
  j -= (uint32_t)u.gd.neps;
  // matching unit: the j-th non-epsilon arc of the smaller side; only the
  // first arc of a label does the label's join
  const View &side = u.joinA ? P.aOut : P.bOut;
  const Grp &g = u.joinA ? u.ga : u.gb;
  const int32_t p = g.begin + g.neps + (int32_t)j;
  const int32_t lab = side.arec[p].x;
  if (p > g.begin + g.neps && side.arec[p - 1].x == lab) return;
  int32_t a0, a1, b0, b1;
  if (u.joinA) {
    bucket(P.aOut, k.qa, p, u.ga.end, lab, a0, a1);
    bucket(P.bOut, k.qb, u.gb.begin + u.gb.neps, u.gb.end, lab, b0, b1);
  } else {
    bucket(P.bOut, k.qb, p, u.gb.end, lab, b0, b1);
    bucket(P.aOut, k.qa, u.ga.begin + u.ga.neps, u.ga.end, lab, a0, a1);
  }
  for (int32_t pa = a0; pa < a1; ++pa) {
    const int32_t ea = P.aOut.perm[pa], ia = P.aOut.olab[pa];
    const uint32_t ta = nbr_of_arc(P.aOut.arec[pa].y);
    const float wa = P.aOut.w[pa];
    for (int32_t pb = b0; pb < b1; ++pb) t_with_d(P, u, pb, ea, ta, 0, ia, wa + P.bOut.w[pb], f);
  }
}

__device__ __forceinline__ bool key_accepts(const Problem3 &P, const Key3 &k) {
  return P.A.accept[k.qa] && P.B.accept[k.qb] && P.D.accept[k.qd];
}

// ---------------------------------------------------------------------------
// preprocessing
// ---------------------------------------------------------------------------

// B state flags: an arc eps:eps (BF_EPS_EPS), an arc y:eps with y != eps
// (BF_EPS_OUT).
__global__ __launch_bounds__(NT) void k3_bflags(DevGraph B, uint32_t *bflags) {
  for (long long e = (long long)blockIdx.x * NT + threadIdx.x; e < B.E;
       e += (long long)gridDim.x * NT) {
    if (B.ol[e] != 0) continue;
    atomicOr(bflags + B.src[e], B.il[e] == 0 ? BF_EPS_EPS : BF_EPS_OUT);
  }
}

// Bucket table of a view: lut[v * stride + l] = {first position of label
// l in group v, first position past it, the first arc's neighbour field
// (0 for an empty bucket), 0}.
__global__ __launch_bounds__(NT) void k3_lut(View v, long long nstates) {
  const long long n = nstates * v.lstride;
  int4 *lut = const_cast<int4 *>(v.lut);
  for (long long x = (long long)blockIdx.x * NT + threadIdx.x; x < n;
       x += (long long)gridDim.x * NT) {
    const uint32_t q = (uint32_t)(x / v.lstride);
    const int32_t l = (int32_t)(x % v.lstride);
    const int4 r = v.srec[2 * (size_t)q];
    int32_t a = r.x, b = r.z;
    while (a < b) {
      const int32_t mid = a + ((b - a) >> 1);
      if (v.arec[mid].x < l) a = mid + 1; else b = mid;
    }
    const int32_t lo = a;
    b = r.z;
    while (a < b) {
      const int32_t mid = a + ((b - a) >> 1);
      if (v.arec[mid].x <= l) a = mid + 1; else b = mid;
    }
    lut[x] = make_int4(lo, a, lo < a ? v.arec[lo].y : 0, 0);
  }
}

// Chain records of B's out-view for the chain jumps of the search: per
// state, up to CHAIN_STEPS steps {n, l0, s0, l1, s1, ...} (CHAIN_INT4
// int4), where step i follows the only arc of the state reached after i
// steps, an arc with input label l_i != epsilon and output epsilon, to s_i.
__global__ __launch_bounds__(NT) void k3_chains(View v, long long nstates, int4 *chain) {
  for (long long q = (long long)blockIdx.x * NT + threadIdx.x; q < nstates;
       q += (long long)gridDim.x * NT) {
    int32_t w[4 * CHAIN_INT4] = {};
    int n = 0;
    uint32_t cur = (uint32_t)q;
#pragma unroll
    for (int k = 0; k < CHAIN_STEPS; ++k) {
      if (n == k) {
        const int4 r = v.srec[2 * (size_t)cur];
        const bool one = r.z - r.x == 1;
        const int2 a = one ? v.arec[r.x] : make_int2(0, 0);
        const int32_t ol = one ? v.olab[r.x] : 1;
        if (one && a.x != 0 && ol == 0) {
          w[1 + 2 * k] = a.x;
          w[2 + 2 * k] = (int32_t)nbr_of_arc(a.y);
          cur = nbr_of_arc(a.y);
          n = k + 1;
        }
      }
    }
    w[0] = n;
    int4 *c = chain + CHAIN_INT4 * q;
#pragma unroll
    for (int k = 0; k < CHAIN_INT4; ++k)
      c[k] = make_int4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
  }
}

// ---------------------------------------------------------------------------
// forward search
// ---------------------------------------------------------------------------

// Start states of one graph into a list (count zeroed by the caller).
__global__ __launch_bounds__(NT) void k3_starts(const uint8_t *flags, int V, int32_t *list,
                                                uint32_t *count) {
  for (long long v0 = (long long)blockIdx.x * NT; v0 < V; v0 += (long long)gridDim.x * NT) {
    const long long v = v0 + threadIdx.x;
    const bool want = v < V && flags[v] != 0;
    const ull m = __ballot(want);
    if (m == 0) continue;
    const int leader = __ffsll(m) - 1;
    uint32_t base = 0;
    if ((int)__lane_id() == leader) base = atomicAdd(count, (uint32_t)__popcll(m));
    base = __shfl(base, leader, WAVE);
    if (want) list[base + __popcll(m & __lanemask_lt())] = (int32_t)v;
  }
}

// Start keys (sa, sb, 0, sd, 0) for every triple of start states: lists of
// A's, B's and D's start states at lists, lists + V_A, lists + V_A + V_B,
// their counts in counts[0..2].
__global__ __launch_bounds__(NT) void k3_seed(Problem3 P, Search3 S, const int32_t *lists,
                                              const uint32_t *counts) {
  const ull na = counts[0], nb = counts[1], nd = counts[2], n = na * nb * nd;
  const int32_t *la = lists, *lb = lists + P.A.V, *ld = lists + P.A.V + P.B.V;
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    bool push = false;
    uint32_t slot = 0;
    if (i < n) {
      const uint32_t qa = (uint32_t)la[i / (nb * nd)], qb = (uint32_t)lb[(i / nd) % nb],
                     qd = (uint32_t)ld[i % nd];
      bool fresh;
      slot = h_insert(P, pack3(P, qa, qb, 0, qd, 0), fresh, &S.sc->overflow);
      push = fresh && slot != NO_SLOT;
    }
    wave_append<uint32_t>(push, slot, S.F, S.fcap, &S.ring[0].fcount, &S.sc->overflow);
  }
}

// Keys one search thread may expand depth-first, one after the other,
// before it hands new keys to the next level.
constexpr int CHAIN3 = 64;

// The chunk list of level l: levels of even and odd number use the two
// halves of the chunk array (ccap entries each), so a level's chunks are
// read while the next level's are written.
__device__ __forceinline__ uint2 *chunks_of(const Search3 &S, int l) {
  return S.chunks + (size_t)(l & 1) * S.ccap;
}

// Sum of v over the wave into *counter (one atomic); every lane of the
// wave takes part.
__device__ __forceinline__ void wave_add(uint32_t v, uint32_t *counter) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  if (__lane_id() == 0 && v) atomicAdd(counter, v);
}

// Chunks of CHUNK3 units of a heavy key into level l's chunk list (counter
// lv = the level's ring slot).
__device__ __forceinline__ void push_chunks(const Search3 &S, Lvl3 *lv, int l, uint32_t slot,
                                            uint32_t n) {
  uint2 *list = chunks_of(S, l);
  const uint32_t nc = (n + CHUNK3 - 1) / CHUNK3;
  const uint32_t c0 = atomicAdd(&lv->ccount, nc);
  for (uint32_t c = 0; c < nc; ++c) {
    if ((ull)c0 + c < S.ccap) list[c0 + c] = make_uint2(slot, c * CHUNK3);
    else atomicOr(&S.sc->overflow, 1u);
  }
}

// The moves of units [u0, u1) of the key in `slot`: every target is looked
// up / inserted and every move recorded as an arc (source slot, target
// slot).  The first new key becomes *cont (its key *cont_key) when the
// thread may go on depth-first (cont not null and none taken yet); other
// new keys join the next frontier.
__device__ __forceinline__ void expand_units(const Problem3 &P, const Search3 &S, uint32_t slot,
                                             const Units3 &u, uint32_t u0, uint32_t u1, Lvl3 *nx,
                                             uint32_t nbase, uint32_t *cont, ull *cont_key) {
  for (uint32_t j = u0; j < u1; ++j)
    for_unit3(P, u, j, [&](ull t, int32_t, int32_t, float, int32_t, int32_t, int32_t) {
      bool fresh;
      const uint32_t ts = h_insert(P, t, fresh, &S.sc->overflow);
      if (ts == NO_SLOT) return;
      wave_append<uint2>(true, make_uint2(slot, ts), S.arcs, S.acap, &S.sc->narcs,
                         &S.sc->overflow);
      bool push = fresh;
      if (fresh && cont && *cont == NO_SLOT) {
        *cont = ts;
        *cont_key = t;
        push = false;
      }
      wave_append<uint32_t>(push, ts, S.F + nbase, (ull)S.fcap - nbase, &nx->fcount,
                            &S.sc->overflow);
    });
}

// Chain jumps.  A key (qa, qb, f1, qd, 0) whose matching move joins the
// one arc of qb (input l != epsilon, output epsilon) with the one arc of
// label l out of qa reaches (qa', qb', 0, qd, 0); along the chain record of
// qb such moves follow each other as long as every key reached again has
// that one matching move (no epsilon output at its A state, one arc of the
// next label).  Beside it a key has at most one more move, the epsilon arc
// of qd when qd has one (a grammar's backoff): it reaches the side key (qa,
// qb, f1, d', 1), since the matching move is a T-arc with output epsilon.
// Hop 0's A bucket is looked up first; the buckets of the later hops (with
// the epsilon counts of their A states) are then loaded together at A
// states guessed to continue hop 0's step, and verified in order (a hop
// whose guessed state was wrong ends the jump).  The keys reached, then the
// side keys, are inserted together (their groups loaded, then one CAS
// each; a key that loses its slot takes the general insert).  The moves of
// the keys this thread inserted, and of the key it started from, are
// recorded as arcs with one atomic; a key another thread inserted is
// expanded by that thread, which records its moves.  New side keys join the
// next frontier.
constexpr int JUMP3 = 8;  // hops per jump

struct Jump3 {
  bool done;       // the jump was taken (else the key is expanded as usual)
  int hops;        // keys reached
  uint32_t fresh;  // of them, inserted by this thread
  uint32_t last;   // slot of the last key reached if this thread inserted it, else NO_SLOT
  ull last_key;
};

// Slots of keys key[i], i in the mask `valid`, inserted if absent (fr[i]):
// all groups loaded, then one CAS per key at the first free slot of its
// group; a key whose group is full or whose slot another key took goes
// through h_insert.  ts[i] = NO_SLOT (and the overflow flag) when the table
// is full.
__device__ __forceinline__ void insert_batch(const Problem3 &P, const Search3 &S,
                                             const ull key[JUMP3], uint32_t valid,
                                             uint32_t ts[JUMP3], bool fr[JUMP3]) {
  uint32_t h[JUMP3], pick[JUMP3];
  // pick[i]: HGROUP + j when slot j of the first group holds the key, j
  // when it is the group's first free slot, 2 HGROUP when neither
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    h[i] = (uint32_t)mix64(key[i]) & P.hmask & ~(HGROUP - 1u);
    pick[i] = 2 * HGROUP;
    if ((valid >> i) & 1u) {
      ull g[HGROUP];
      load_group(P, h[i], g);
#pragma unroll
      for (int j = HGROUP - 1; j >= 0; --j)
        if (g[j] == EMPTY3) pick[i] = (uint32_t)j;
#pragma unroll
      for (int j = HGROUP - 1; j >= 0; --j)
        if (g[j] == key[i]) pick[i] = HGROUP + (uint32_t)j;
    }
  }
  ull old[JUMP3];
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    old[i] = 0;
    if (((valid >> i) & 1u) && pick[i] < HGROUP)
      old[i] = atomicCAS(P.tab + h[i] + pick[i], EMPTY3, key[i]);
  }
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    ts[i] = NO_SLOT;
    fr[i] = false;
    if ((valid >> i) & 1u) {
      if (pick[i] >= HGROUP && pick[i] < 2 * HGROUP) {
        ts[i] = h[i] + pick[i] - HGROUP;
      } else if (pick[i] < HGROUP && old[i] == EMPTY3) {
        ts[i] = h[i] + pick[i];
        fr[i] = true;
      } else if (pick[i] < HGROUP && old[i] == key[i]) {
        ts[i] = h[i] + pick[i];
      } else {
        ts[i] = h_insert(P, key[i], fr[i], &S.sc->overflow);
      }
    }
  }
}

__device__ __forceinline__ Jump3 jump3(const Problem3 &P, const Search3 &S, uint32_t slot,
                                       const Units3 &u, int max_hops, Lvl3 *nx,
                                       uint32_t nbase) {
  Jump3 r;
  r.done = false;
  const Key3 &k = u.k;
  if (!P.bOut.chain || !P.aOut.lut || max_hops < 1) return r;
  if (k.f2 != 0 || u.nae != 0 || u.gb.neps != 0 || u.gd.neps > 1 ||
      u.gb.end - u.gb.begin != 1)
    return r;
  const int4 *cr = P.bOut.chain + CHAIN_INT4 * (size_t)k.qb;
  int32_t cw[4 * CHAIN_INT4];
#pragma unroll
  for (int q = 0; q < CHAIN_INT4; ++q) {
    const int4 c = cr[q];
    cw[4 * q] = c.x;
    cw[4 * q + 1] = c.y;
    cw[4 * q + 2] = c.z;
    cw[4 * q + 3] = c.w;
  }
  // the target of qd's epsilon arc, if it has one
  const bool side = u.gd.neps == 1;
  const uint32_t dd = side ? nbr_of_arc(P.dOut.arec[u.gd.begin].y) : 0u;
  int n = cw[0];
  if (n > max_hops) n = max_hops;
  if (n > JUMP3) n = JUMP3;
  const uint32_t stride = (uint32_t)P.aOut.lstride, VA = (uint32_t)P.A.V;
  if (n < 1 || (uint32_t)cw[1] >= stride) return r;
  const int4 *lut = P.aOut.lut;
  const int4 b0 = lut[(size_t)k.qa * stride + (uint32_t)cw[1]];
  if (b0.y - b0.x != 1) return r;
  uint32_t qa[JUMP3 + 1];  // A state of the key reached after i hops, i <= m
  qa[0] = k.qa;
  qa[1] = nbr_of_arc(b0.z);
  const uint32_t step = qa[1] - qa[0];  // modulo 2^32
  int4 bk[JUMP3];
  int32_t ek[JUMP3];
#pragma unroll
  for (int i = 1; i < JUMP3; ++i) {
    const uint32_t g = qa[0] + (uint32_t)i * step;
    const uint32_t lab = (uint32_t)cw[1 + 2 * i];
    bk[i] = make_int4(0, 0, 0, 0);
    ek[i] = 1;
    if (i < n && g < VA && lab < stride) {
      bk[i] = lut[(size_t)g * stride + lab];
      ek[i] = P.aOut.srec[2 * (size_t)g].y;
    }
  }
  int m = 1;  // hops taken
#pragma unroll
  for (int i = 1; i < JUMP3; ++i)
    if (m == i && i < n && qa[0] + (uint32_t)i * step == qa[i] && bk[i].y - bk[i].x == 1 &&
        ek[i] == 0) {
      qa[i + 1] = nbr_of_arc(bk[i].z);
      m = i + 1;
    }
  // a segment of the keys that lead to the last one (its slot taken now,
  // so the atomic returns during the inserts)
  const uint32_t sidx = (S.segs && m >= 2) ? atomicAdd(&S.sc->nseg, 1u) : NO_SLOT;
  // the keys reached, (qa[i + 1], s_i, 0, qd, 0) for i < m
  ull key[JUMP3];
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    key[i] = pack3(P, qa[i + 1 <= m ? i + 1 : m], (uint32_t)cw[2 + 2 * i], 0, k.qd, 0);
  uint32_t ts[JUMP3];
  bool fr[JUMP3];
  insert_batch(P, S, key, (1u << m) - 1u, ts, fr);
  // the side keys of the hops' sources, (qa[i], s_(i-1) (qb for i = 0),
  // f1 of the source, d', 1) for i < m
  ull skey[JUMP3];
  uint32_t sts[JUMP3];
  bool sfr[JUMP3];
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    skey[i] = pack3(P, qa[i <= m ? i : m], i == 0 ? k.qb : (uint32_t)cw[2 * i],
                    i == 0 ? k.f1 : 0u, dd, 1);
  insert_batch(P, S, skey, side ? (1u << m) - 1u : 0u, sts, sfr);
  r.done = true;
  r.hops = m;
  r.fresh = 0;
  r.last = NO_SLOT;
  r.last_key = 0;
  bool full = false;
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    if (i < m) {
      full = full || ts[i] == NO_SLOT || (side && sts[i] == NO_SLOT);
      r.fresh += fr[i] ? 1u : 0u;
    }
  if (full) return r;  // the table is full: the search starts again
  // the moves of the hops' sources this thread owns: the start key, and
  // the keys it inserted before the last
  bool own[JUMP3];
  uint32_t nown = 0, nside = 0;
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    own[i] = i < m && (i == 0 || fr[i - 1]);
    nown += own[i] ? 1u : 0u;
    nside += (i < m && side && sfr[i]) ? 1u : 0u;
  }
  const uint32_t per = side ? 2u : 1u;
  const ull base = atomicAdd(&S.sc->narcs, nown * per);
  uint32_t o = 0;
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    if (own[i]) {
      const uint32_t src = i == 0 ? slot : ts[i - 1];
      if (base + o + per <= S.acap) {
        S.arcs[base + o] = make_uint2(src, ts[i]);
        if (side) S.arcs[base + o + 1] = make_uint2(src, sts[i]);
      } else {
        atomicOr(&S.sc->overflow, 1u);
      }
      o += per;
    }
  if (sidx < S.scap) {
    uint32_t *sg = S.segs + 8 * (size_t)sidx;
#pragma unroll
    for (int i = 0; i < JUMP3; ++i)
      if (i < m) sg[i] = i == 0 ? slot : ts[i - 1];
#pragma unroll
    for (int i = 0; i < JUMP3; ++i)
      if (i + 1 == m) S.seg_of[ts[i]] = sidx << 4 | (uint32_t)m;
  }
  // new side keys join the next frontier
  if (nside) {
    const uint32_t fb = atomicAdd(&nx->fcount, nside);
    uint32_t q = 0;
#pragma unroll
    for (int i = 0; i < JUMP3; ++i)
      if (i < m && side && sfr[i]) {
        const ull pos = (ull)fb + q;
        if (pos < (ull)S.fcap - nbase) S.F[nbase + pos] = sts[i];
        else atomicOr(&S.sc->overflow, 1u);
        ++q;
      }
  }
  // the last key goes on the walk if this thread inserted it
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    if (i + 1 == m && fr[i]) {
      r.last_key = key[i];
      r.last = ts[i];
    }
  return r;
}

// A thread's depth-first walk from `key` (in `slot`): a key with at most
// WALK3 units is expanded at once (a chain of one-move keys by a jump) and
// the walk goes on with the first new key it reached (up to CHAIN3 keys); a
// heavier key is cut into chunks for the chunk list `heavy_to`.  Every
// other new key joins the next frontier.  Returns the number of keys the
// walk inserted and did not put in a frontier.
__device__ __forceinline__ uint32_t walk_fwd(const Problem3 &P, const Search3 &S, uint32_t slot,
                                             ull key, Lvl3 *nx, uint32_t nbase, Lvl3 *heavy_to,
                                             int heavy_l) {
  uint32_t went = 0;
  for (int depth = 0; depth < CHAIN3; ++depth) {
    const Units3 u = units_of(P, key);
    const uint32_t n = nunits(u);
    if (n > WALK3) {
      push_chunks(S, heavy_to, heavy_l, slot, n);
      return went;
    }
    // the key reached last must still be expanded within the budget
    const Jump3 j = jump3(P, S, slot, u, CHAIN3 - 1 - depth, nx, nbase);
    if (j.done) {
      went += j.fresh;
      if (j.last == NO_SLOT) return went;
      depth += j.hops - 1;
      slot = j.last;
      key = j.last_key;
      continue;
    }
    uint32_t cont = NO_SLOT;
    ull cont_key = 0;
    expand_units(P, S, slot, u, 0, n, nx, nbase, depth + 1 < CHAIN3 ? &cont : nullptr,
                 &cont_key);
    if (cont == NO_SLOT) return went;
    ++went;
    slot = cont;
    key = cont_key;
  }
  return went;
}

// Level l of the forward search: frontier entries [fbase, fbase + fcount)
// of ring[l % 3], each the start of a depth-first walk; heavy keys met go to
// this level's chunks (k3_fwd_chunks, next).  Block 0 publishes the next
// level's frontier base and clears the ring slot of level l + 2.
__global__ __launch_bounds__(NT) void k3_fwd(Problem3 P, Search3 S, int l) {
  const Lvl3 cur = S.ring[l % 3];
  Lvl3 *nx = &S.ring[(l + 1) % 3];
  const uint32_t nbase = cur.fbase + cur.fcount;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    nx->fbase = nbase;
    Lvl3 *done = &S.ring[(l + 2) % 3];
    done->fcount = 0;
    done->ccount = 0;
    if (cur.fcount || cur.ccount) S.sc->levels = (uint32_t)l + 1;
  }
  uint32_t went = 0;
  if (!S.sc->overflow)
    for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i < cur.fcount; i += (ull)gridDim.x * NT) {
      const uint32_t slot = S.F[cur.fbase + i];
      went += walk_fwd(P, S, slot, P.tab[slot], nx, nbase, &S.ring[l % 3], l);
    }
  wave_add(went, &S.sc->ncont);
}

// Units [u0, u1) of the key in `slot` when they are all arcs of its B
// state with input epsilon (a lexicon root's word entries), each with at
// most one D arc for its output (or none needed): their arc records, D
// buckets and targets are loaded together and the targets inserted
// together, the moves recorded with one atomic; the first new target
// becomes *cont, the others join the next frontier.  Returns false (nothing
// done) when the units do not have that shape.
__device__ __forceinline__ bool expand_beps(const Problem3 &P, const Search3 &S, uint32_t slot,
                                            const Units3 &u, uint32_t u0, uint32_t u1,
                                            Lvl3 *nx, uint32_t nbase, uint32_t *cont,
                                            ull *cont_key) {
  static_assert(CHUNK3 <= JUMP3, "a chunk's units fit one batch");
  const Key3 &k = u.k;
  if (!P.dOut.lut || u1 - u0 > (uint32_t)JUMP3 || u0 < u.nae ||
      u1 > u.nae + (uint32_t)u.gb.neps)
    return false;
  const uint32_t tf1 = u.ga.neps > 0 ? 1u : 0u;  // epsOutA(qa)
  const uint32_t dstride = (uint32_t)P.dOut.lstride;
  int32_t z[JUMP3];
  uint32_t tb[JUMP3];
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    z[i] = 0;
    tb[i] = 0;
    if (u0 + (uint32_t)i < u1) {
      const int32_t p = u.gb.begin + (int32_t)(u0 - u.nae) + i;
      z[i] = P.bOut.olab[p];
      tb[i] = nbr_of_arc(P.bOut.arec[p].y);
    }
  }
  int4 db[JUMP3];
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    db[i] = make_int4(0, 0, 0, 0);
    if (u0 + (uint32_t)i < u1 && z[i] != 0 && (uint32_t)z[i] < dstride)
      db[i] = P.dOut.lut[(size_t)k.qd * dstride + (uint32_t)z[i]];
  }
  // a unit with several D arcs for its output takes the general path
  uint32_t valid = 0;
  ull key[JUMP3];
#pragma unroll
  for (int i = 0; i < JUMP3; ++i) {
    key[i] = 0;
    if (u0 + (uint32_t)i >= u1) continue;
    if (z[i] == 0) {
      if (k.f2 == 0) {  // a T-arc with output epsilon, alone
        key[i] = pack3(P, k.qa, tb[i], tf1, k.qd, 0);
        valid |= 1u << i;
      }
    } else if (db[i].y - db[i].x == 1) {
      key[i] = pack3(P, k.qa, tb[i], tf1, nbr_of_arc(db[i].z), 0);
      valid |= 1u << i;
    } else if (db[i].y - db[i].x > 1) {
      return false;
    }
  }
  uint32_t ts[JUMP3];
  bool fr[JUMP3];
  insert_batch(P, S, key, valid, ts, fr);
  uint32_t nv = 0, nnew = 0;
  bool full = false;
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    if ((valid >> i) & 1u) {
      ++nv;
      full = full || ts[i] == NO_SLOT;
    }
  if (full) return true;  // the table is full: the search starts again
  if (nv) {
    const ull base = atomicAdd(&S.sc->narcs, nv);
    uint32_t o = 0;
#pragma unroll
    for (int i = 0; i < JUMP3; ++i)
      if ((valid >> i) & 1u) {
        if (base + o < S.acap) S.arcs[base + o] = make_uint2(slot, ts[i]);
        else atomicOr(&S.sc->overflow, 1u);
        ++o;
      }
  }
  // the first new target goes on the walk, the others to the next frontier
#pragma unroll
  for (int i = 0; i < JUMP3; ++i)
    if (((valid >> i) & 1u) && fr[i]) {
      if (*cont == NO_SLOT) {
        *cont = ts[i];
        *cont_key = key[i];
        fr[i] = false;
      } else {
        ++nnew;
      }
    }
  if (nnew) {
    const uint32_t fb = atomicAdd(&nx->fcount, nnew);
    uint32_t q = 0;
#pragma unroll
    for (int i = 0; i < JUMP3; ++i)
      if (((valid >> i) & 1u) && fr[i]) {
        const ull pos = (ull)fb + q;
        if (pos < (ull)S.fcap - nbase) S.F[nbase + pos] = ts[i];
        else atomicOr(&S.sc->overflow, 1u);
        ++q;
      }
  }
  return true;
}

// The chunks of level l: CHUNK3 units each, then a depth-first walk from
// the first new key; heavy keys met on the walk go to the next level's
// chunks.
__global__ __launch_bounds__(NT) void k3_fwd_chunks(Problem3 P, Search3 S, int l) {
  const Lvl3 cur = S.ring[l % 3];
  Lvl3 *nx = &S.ring[(l + 1) % 3];
  const uint32_t nbase = cur.fbase + cur.fcount;
  const uint32_t nch = S.sc->overflow ? 0 : (cur.ccount < S.ccap ? cur.ccount : S.ccap);
  const uint2 *list = chunks_of(S, l);
  uint32_t went = 0;
  for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i < nch; i += (ull)gridDim.x * NT) {
    const uint2 c = list[i];
    const Units3 u = units_of(P, P.tab[c.x]);
    const uint32_t n = nunits(u);
    const uint32_t u1 = c.y + CHUNK3 < n ? c.y + CHUNK3 : n;
    uint32_t cont = NO_SLOT;
    ull cont_key = 0;
    if (!expand_beps(P, S, c.x, u, c.y, u1, nx, nbase, &cont, &cont_key))
      expand_units(P, S, c.x, u, c.y, u1, nx, nbase, &cont, &cont_key);
    if (cont != NO_SLOT) went += 1 + walk_fwd(P, S, cont, cont_key, nx, nbase, nx, l + 1);
  }
  wave_add(went, &S.sc->ncont);
}

// ---------------------------------------------------------------------------
// backward search over the recorded arcs
// ---------------------------------------------------------------------------

// In-arcs grouped by target without atomics: the arcs as (target, source)
// pairs, sorted by target (a radix sort); then each run of one target marks
// its first position (run start) and, at its last, its length (the target's
// in-degree); a scan of the in-degrees gives the offsets, and the sorted
// sources are the in-arc lists.
__global__ __launch_bounds__(NT) void k3_arc_keys(const uint2 *arcs, ull narcs, ull *key,
                                                  int32_t *src) {
  for (ull e = (ull)blockIdx.x * NT + threadIdx.x; e < narcs; e += (ull)gridDim.x * NT) {
    const uint2 a = arcs[e];
    key[e] = a.y;
    src[e] = (int32_t)a.x;
  }
}

__global__ __launch_bounds__(NT) void k3_run_starts(const ull *key, ull narcs,
                                                    uint32_t *first) {
  for (ull e = (ull)blockIdx.x * NT + threadIdx.x; e < narcs; e += (ull)gridDim.x * NT)
    if (e == 0 || key[e] != key[e - 1]) first[key[e]] = (uint32_t)e;
}

__global__ __launch_bounds__(NT) void k3_run_ends(const ull *key, ull narcs,
                                                  const uint32_t *first, uint32_t *indeg) {
  for (ull e = (ull)blockIdx.x * NT + threadIdx.x; e < narcs; e += (ull)gridDim.x * NT)
    if (e + 1 == narcs || key[e] != key[e + 1]) indeg[key[e]] = (uint32_t)(e + 1) - first[key[e]];
}

__device__ __forceinline__ bool claim_bit(uint32_t *bm, uint32_t s) {
  const uint32_t bit = 1u << (s & 31u);
  if (bm[s >> 5] & bit) return false;
  return (atomicOr(bm + (s >> 5), bit) & bit) == 0;
}

// Accepting keys seed the backward search (level 0 of its ring).
__global__ __launch_bounds__(NT) void k3_seed_bwd(Problem3 P, Search3 S) {
  const ull H = (ull)P.hmask + 1;
  for (ull i0 = (ull)blockIdx.x * NT; i0 < H; i0 += (ull)gridDim.x * NT) {
    const ull s = i0 + threadIdx.x;
    bool push = false;
    if (s < H) {
      const ull k = P.tab[s];
      if (k != EMPTY3 && key_accepts(P, unpack3(P, k))) {
        atomicOr(P.coacc + (s >> 5), 1u << (s & 31u));
        push = true;
      }
    }
    wave_append<uint32_t>(push, (uint32_t)s, S.F, S.fcap, &S.ring[0].fcount, &S.sc->overflow);
  }
}

// Sources of in-arcs [p0, p1): each one claimed becomes *cont (the first,
// when allowed) or joins the next frontier.
__device__ __forceinline__ void bwd_range(const Problem3 &P, const Search3 &S, uint32_t p0,
                                          uint32_t p1, Lvl3 *nx, uint32_t nbase,
                                          uint32_t *cont) {
  for (uint32_t p = p0; p < p1; ++p) {
    const uint32_t u = P.in_src[p];
    bool push = claim_bit(P.coacc, u);
    if (push && cont && *cont == NO_SLOT) {
      *cont = u;
      push = false;
    }
    wave_append<uint32_t>(push, u, S.F + nbase, (ull)S.fcap - nbase, &nx->fcount,
                          &S.sc->overflow);
  }
}

// A slot into the next frontier (one atomic).
__device__ __forceinline__ void push_one(const Search3 &S, Lvl3 *nx, uint32_t nbase, uint32_t u) {
  const uint32_t pos = atomicAdd(&nx->fcount, 1u);
  if ((ull)pos < (ull)S.fcap - nbase) S.F[nbase + pos] = u;
  else atomicOr(&S.sc->overflow, 1u);
}

// The keys of chain segment sg (see Search3), which lead to a key found
// co-accessible, are claimed together (their bitmap words loaded, then one
// atomic each for the unclaimed).  A newly claimed key other than the first
// that has in-arcs besides the one from its predecessor on the segment
// joins the next frontier (its in-arcs are walked from there); the first
// key, if newly claimed, is returned to walk on from (cont allowed) or
// joins the next frontier.  *went counts the claimed keys not put in a
// frontier.
__device__ __forceinline__ uint32_t claim_segment(const Problem3 &P, const Search3 &S,
                                                  uint32_t sg, Lvl3 *nx, uint32_t nbase,
                                                  bool cont, uint32_t *went) {
  const uint32_t n = sg & 15u;
  const uint32_t *seg = S.segs + 8 * (size_t)(sg >> 4);
  uint32_t u[JUMP3], w[JUMP3];
#pragma unroll
  for (int j = 0; j < JUMP3; ++j) u[j] = (uint32_t)j < n ? seg[j] : 0u;
#pragma unroll
  for (int j = 0; j < JUMP3; ++j) w[j] = (uint32_t)j < n ? P.coacc[u[j] >> 5] : ~0u;
  bool fr[JUMP3];
#pragma unroll
  for (int j = 0; j < JUMP3; ++j) {
    const uint32_t bit = 1u << (u[j] & 31u);
    fr[j] = (uint32_t)j < n && !(w[j] & bit) && (atomicOr(P.coacc + (u[j] >> 5), bit) & bit) == 0;
  }
  uint32_t d[JUMP3];
#pragma unroll
  for (int j = 1; j < JUMP3; ++j) d[j] = fr[j] ? P.in_off[u[j] + 1] - P.in_off[u[j]] : 1u;
#pragma unroll
  for (int j = 1; j < JUMP3; ++j)
    if (fr[j]) {
      if (d[j] != 1u) push_one(S, nx, nbase, u[j]);
      else ++*went;
    }
  if (!fr[0]) return NO_SLOT;
  if (cont) return u[0];
  push_one(S, nx, nbase, u[0]);
  return NO_SLOT;
}

// Depth-first backward walk from slot v (as walk_fwd, over in-arcs; a key
// that ends a chain segment has the segment's keys claimed first).
__device__ __forceinline__ uint32_t walk_bwd(const Problem3 &P, const Search3 &S, uint32_t v,
                                             Lvl3 *nx, uint32_t nbase, Lvl3 *heavy_to,
                                             int heavy_l) {
  uint32_t went = 0;
  for (int depth = 0; depth < CHAIN3; ++depth) {
    const uint32_t p0 = P.in_off[v], p1 = P.in_off[v + 1];
    const uint32_t sg = S.seg_of ? S.seg_of[v] : NO_SLOT;
    uint32_t cont = NO_SLOT;
    if (sg != NO_SLOT) cont = claim_segment(P, S, sg, nx, nbase, depth + 1 < CHAIN3, &went);
    if (p1 - p0 > WALK3) {
      if (cont != NO_SLOT) push_one(S, nx, nbase, cont);
      push_chunks(S, heavy_to, heavy_l, v, p1 - p0);
      return went;
    }
    bwd_range(P, S, p0, p1, nx, nbase, depth + 1 < CHAIN3 ? &cont : nullptr);
    if (cont == NO_SLOT) return went;
    ++went;
    v = cont;
  }
  return went;
}

__global__ __launch_bounds__(NT) void k3_bwd(Problem3 P, Search3 S, int l) {
  const Lvl3 cur = S.ring[l % 3];
  Lvl3 *nx = &S.ring[(l + 1) % 3];
  const uint32_t nbase = cur.fbase + cur.fcount;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    nx->fbase = nbase;
    Lvl3 *done = &S.ring[(l + 2) % 3];
    done->fcount = 0;
    done->ccount = 0;
    if (cur.fcount || cur.ccount) S.sc->levels = (uint32_t)l + 1;
  }
  uint32_t went = 0;
  if (!S.sc->overflow)
    for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i < cur.fcount; i += (ull)gridDim.x * NT)
      went += walk_bwd(P, S, S.F[cur.fbase + i], nx, nbase, &S.ring[l % 3], l);
  wave_add(went, &S.sc->ncont);
}

__global__ __launch_bounds__(NT) void k3_bwd_chunks(Problem3 P, Search3 S, int l) {
  const Lvl3 cur = S.ring[l % 3];
  Lvl3 *nx = &S.ring[(l + 1) % 3];
  const uint32_t nbase = cur.fbase + cur.fcount;
  const uint32_t nch = S.sc->overflow ? 0 : (cur.ccount < S.ccap ? cur.ccount : S.ccap);
  const uint2 *list = chunks_of(S, l);
  uint32_t went = 0;
  for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i < nch; i += (ull)gridDim.x * NT) {
    const uint2 c = list[i];
    const uint32_t p0 = P.in_off[c.x] + c.y, pe = P.in_off[c.x + 1];
    const uint32_t p1 = p0 + CHUNK3 < pe ? p0 + CHUNK3 : pe;
    uint32_t cont = NO_SLOT;
    bwd_range(P, S, p0, p1, nx, nbase, &cont);
    if (cont != NO_SLOT) went += 1 + walk_bwd(P, S, cont, nx, nbase, nx, l + 1);
  }
  wave_add(went, &S.sc->ncont);
}

// ---------------------------------------------------------------------------
// trim, numbering, count, fill
// ---------------------------------------------------------------------------

// Trim keys (in the set and co-accessible) with their slots.  Each
// workgroup takes COL_ITEMS x NT consecutive slots per round and appends
// its keys with one atomic (a workgroup scan places them).
constexpr int COL_ITEMS = 8;

__global__ __launch_bounds__(NT) void k3_collect(Problem3 P, ull *keys, int32_t *slots,
                                                 uint32_t *count, uint32_t cap,
                                                 uint32_t *overflow) {
  __shared__ uint32_t s_w[NWAVES];
  __shared__ uint32_t s_base;
  const ull H = (ull)P.hmask + 1;
  const ull tile = (ull)NT * COL_ITEMS;
  for (ull b0 = (ull)blockIdx.x * tile; b0 < H; b0 += (ull)gridDim.x * tile) {
    ull kv[COL_ITEMS];
    uint32_t want = 0, c = 0;
#pragma unroll
    for (int r = 0; r < COL_ITEMS; ++r) {
      const ull sl = b0 + (ull)threadIdx.x * COL_ITEMS + r;
      kv[r] = EMPTY3;
      if (sl < H) {
        kv[r] = P.tab[sl];
        if (kv[r] != EMPTY3 && ((P.coacc[sl >> 5] >> (sl & 31u)) & 1u)) {
          want |= 1u << r;
          ++c;
        }
      }
    }
    uint32_t total;
    const uint32_t off = block_excl_scan<uint32_t>(c, s_w, total);
    if (threadIdx.x == 0) s_base = total ? atomicAdd(count, total) : 0u;
    __syncthreads();
    uint32_t pos = s_base + off;
#pragma unroll
    for (int r = 0; r < COL_ITEMS; ++r)
      if (want & (1u << r)) {
        if (pos < cap) {
          keys[pos] = kv[r];
          slots[pos] = (int32_t)(b0 + (ull)threadIdx.x * COL_ITEMS + r);
        } else {
          atomicOr(overflow, 1u);
        }
        ++pos;
      }
    __syncthreads();  // s_base is rewritten next round
  }
}

// id_of[slot] = rank of the slot's key among the trim keys; units of every
// state of C; states with more than LIGHT3 units listed as heavy.
__global__ __launch_bounds__(NT) void k3_ids(Problem3 P, const ull *keys, const int32_t *slots,
                                             uint32_t n, int32_t *id_of, uint32_t *units,
                                             uint32_t *heavy, uint32_t *nheavy) {
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    uint32_t nu = 0;
    if (i < n) {
      id_of[slots[i]] = (int32_t)i;
      nu = nunits(units_of(P, keys[i]));
      units[i] = nu;
    }
    wave_append<uint32_t>(nu > LIGHT3, (uint32_t)i, heavy, n, nheavy, nheavy + 1);
  }
}

__device__ __forceinline__ int32_t id_of_key(const Problem3 &P, ull t) {
  const uint32_t s = h_find(P, t);
  return s == NO_SLOT ? -1 : P.id_of[s];
}

// Kept arcs of unit j of state i, written from position pos (FILL) or
// counted.
template <bool FILL>
__device__ __forceinline__ uint32_t out_unit(const Problem3 &P, const Units3 &st, uint32_t i,
                                             uint32_t j, uint32_t pos, const OutGraph3 &O) {
  uint32_t c = 0;
  for_unit3(P, st, j, [&](ull t, int32_t il, int32_t ol, float w, int32_t a, int32_t b, int32_t d) {
    const int32_t id = id_of_key(P, t);
    if (id < 0) return;
    if (FILL) {
      const uint32_t q = pos + c;
      O.src[q] = (int32_t)i;
      O.dst[q] = id;
      O.il[q] = il;
      O.ol[q] = ol;
      O.w[q] = w;
      if (O.arc_a) O.arc_a[q] = a;
      if (O.arc_b) O.arc_b[q] = b;
      if (O.arc_d) O.arc_d[q] = d;
    }
    ++c;
  });
  return c;
}

// Light states: one thread each, every unit in turn (counts per unit, or
// the arcs at each unit's position).
template <bool FILL>
__global__ __launch_bounds__(NT) void k3_out_light(Problem3 P, const ull *keys,
                                                   const uint32_t *ustart, uint32_t n,
                                                   uint32_t *ucnt, const uint32_t *uoff,
                                                   OutGraph3 O) {
  for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i < n; i += (ull)gridDim.x * NT) {
    const uint32_t u0 = ustart[i], nu = ustart[i + 1] - u0;
    if (nu > LIGHT3) continue;
    const Units3 st = units_of(P, keys[i]);
    for (uint32_t j = 0; j < nu; ++j) {
      const uint32_t c = out_unit<FILL>(P, st, (uint32_t)i, j, FILL ? uoff[u0 + j] : 0u, O);
      if (!FILL) ucnt[u0 + j] = c;
    }
  }
}

// Heavy states: one workgroup each, its threads taking the units in turn.
template <bool FILL>
__global__ __launch_bounds__(NT) void k3_out_heavy(Problem3 P, const ull *keys,
                                                   const uint32_t *ustart, const uint32_t *heavy,
                                                   const uint32_t *nheavy, uint32_t *ucnt,
                                                   const uint32_t *uoff, OutGraph3 O) {
  const uint32_t nh = *nheavy;
  for (uint32_t h = blockIdx.x; h < nh; h += gridDim.x) {
    const uint32_t i = heavy[h];
    const uint32_t u0 = ustart[i], nu = ustart[i + 1] - u0;
    const Units3 st = units_of(P, keys[i]);
    for (uint32_t j = threadIdx.x; j < nu; j += NT) {
      const uint32_t c = out_unit<FILL>(P, st, i, j, FILL ? uoff[u0 + j] : 0u, O);
      if (!FILL) ucnt[u0 + j] = c;
    }
  }
}

__global__ __launch_bounds__(NT) void k3_fill_states(Problem3 P, const ull *keys,
                                                     const uint32_t *ustart, uint32_t n,
                                                     const uint32_t *uoff, uint32_t narcs,
                                                     OutGraph3 O) {
  for (ull i = (ull)blockIdx.x * NT + threadIdx.x; i <= n; i += (ull)gridDim.x * NT) {
    if (i == n) {
      O.arc_offset[n] = (int32_t)narcs;
      continue;
    }
    const Key3 k = unpack3(P, keys[i]);
    O.arc_offset[i] = (int32_t)uoff[ustart[i]];
    O.start[i] = (k.f1 == 0 && k.f2 == 0 && P.A.start[k.qa] && P.B.start[k.qb] &&
                  P.D.start[k.qd]) ? 1 : 0;
    O.accept[i] = key_accepts(P, k) ? 1 : 0;
    if (O.key_a) O.key_a[i] = (int32_t)k.qa;
    if (O.key_b) O.key_b[i] = (int32_t)k.qb;
    if (O.key_fab) O.key_fab[i] = (uint8_t)k.f1;
    if (O.key_d) O.key_d[i] = (int32_t)k.qd;
    if (O.key_f) O.key_f[i] = (uint8_t)k.f2;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

hipError_t launch3_bflags(const DevGraph &B, uint32_t *bflags, hipStream_t s) {
  if (B.E) k3_bflags<<<grid3((size_t)B.E), NT, 0, s>>>(B, bflags);
  return hipGetLastError();
}

hipError_t launch3_starts(const DevGraph &A, const DevGraph &B, const DevGraph &D,
                          int32_t *lists, uint32_t *counts, hipStream_t s) {
  k3_starts<<<grid3((size_t)A.V, 1024), NT, 0, s>>>(A.start, A.V, lists, counts);
  k3_starts<<<grid3((size_t)B.V, 1024), NT, 0, s>>>(B.start, B.V, lists + A.V, counts + 1);
  k3_starts<<<grid3((size_t)D.V, 1024), NT, 0, s>>>(D.start, D.V, lists + A.V + B.V, counts + 2);
  return hipGetLastError();
}

hipError_t launch3_seed(const Problem3 &P, const Search3 &S, const int32_t *lists,
                        const uint32_t *counts, hipStream_t s) {
  k3_seed<<<64, NT, 0, s>>>(P, S, lists, counts);
  return hipGetLastError();
}

hipError_t launch3_level(const Problem3 &P, const Search3 &S, bool forward, int l,
                         hipStream_t s) {
  constexpr unsigned GRID = 1024;
  if (forward) {
    k3_fwd<<<GRID, NT, 0, s>>>(P, S, l);
    k3_fwd_chunks<<<GRID, NT, 0, s>>>(P, S, l);
  } else {
    k3_bwd<<<GRID, NT, 0, s>>>(P, S, l);
    k3_bwd_chunks<<<GRID, NT, 0, s>>>(P, S, l);
  }
  return hipGetLastError();
}

hipError_t launch3_arc_keys(const uint2 *arcs, unsigned long long narcs, unsigned long long *key,
                            int32_t *src, hipStream_t s) {
  if (!narcs) return hipSuccess;
  k3_arc_keys<<<grid3((size_t)narcs), NT, 0, s>>>(arcs, narcs, key, src);
  return hipGetLastError();
}

hipError_t launch3_in_degrees(const unsigned long long *key, unsigned long long narcs,
                              uint32_t *first, uint32_t *indeg, hipStream_t s) {
  if (!narcs) return hipSuccess;
  k3_run_starts<<<grid3((size_t)narcs), NT, 0, s>>>(key, narcs, first);
  k3_run_ends<<<grid3((size_t)narcs), NT, 0, s>>>(key, narcs, first, indeg);
  return hipGetLastError();
}

hipError_t launch3_chains(const View &v, long long nstates, int4 *chain, hipStream_t s) {
  if (nstates > 0) k3_chains<<<grid3((size_t)nstates), NT, 0, s>>>(v, nstates, chain);
  return hipGetLastError();
}

hipError_t launch3_lut(const View &v, long long nstates, hipStream_t s) {
  const long long n = nstates * v.lstride;
  if (n > 0) k3_lut<<<grid3((size_t)n, 8192), NT, 0, s>>>(v, nstates);
  return hipGetLastError();
}

hipError_t launch3_seed_bwd(const Problem3 &P, const Search3 &S, hipStream_t s) {
  k3_seed_bwd<<<grid3((size_t)P.hmask + 1, 8192), NT, 0, s>>>(P, S);
  return hipGetLastError();
}

hipError_t launch3_collect(const Problem3 &P, unsigned long long *keys, int32_t *slots,
                           uint32_t *count, uint32_t cap, uint32_t *overflow, hipStream_t s) {
  const size_t tiles = ((size_t)P.hmask + 1 + (size_t)NT * COL_ITEMS - 1) / ((size_t)NT * COL_ITEMS);
  k3_collect<<<(unsigned)(tiles < 4096 ? tiles : 4096), NT, 0, s>>>(P, keys, slots, count, cap,
                                                                   overflow);
  return hipGetLastError();
}

hipError_t launch3_ids(const Problem3 &P, const unsigned long long *keys, const int32_t *slots,
                       uint32_t n, int32_t *id_of, uint32_t *units, uint32_t *heavy,
                       uint32_t *nheavy, hipStream_t s) {
  if (n) k3_ids<<<grid3(n), NT, 0, s>>>(P, keys, slots, n, id_of, units, heavy, nheavy);
  return hipGetLastError();
}

hipError_t launch3_count(const Problem3 &P, const unsigned long long *keys,
                         const uint32_t *ustart, uint32_t n, const uint32_t *heavy,
                         const uint32_t *nheavy, uint32_t *ucnt, hipStream_t s) {
  if (!n) return hipSuccess;
  const OutGraph3 none = {};
  k3_out_light<false><<<grid3(n, 16384), NT, 0, s>>>(P, keys, ustart, n, ucnt, nullptr, none);
  k3_out_heavy<false><<<1024, NT, 0, s>>>(P, keys, ustart, heavy, nheavy, ucnt, nullptr, none);
  return hipGetLastError();
}

hipError_t launch3_fill(const Problem3 &P, const unsigned long long *keys, const uint32_t *ustart,
                        uint32_t n, const uint32_t *heavy, const uint32_t *nheavy,
                        const uint32_t *uoff, uint32_t narcs, const OutGraph3 &O,
                        hipStream_t s) {
  if (n) {
    k3_out_light<true><<<grid3(n, 16384), NT, 0, s>>>(P, keys, ustart, n, nullptr, uoff, O);
    k3_out_heavy<true><<<1024, NT, 0, s>>>(P, keys, ustart, heavy, nheavy, nullptr, uoff, O);
  }
  k3_fill_states<<<grid3((size_t)n + 1, 8192), NT, 0, s>>>(P, keys, ustart, n, uoff, narcs, O);
  return hipGetLastError();
}

}  // namespace fstc
