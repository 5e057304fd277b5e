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

__global__ __launch_bounds__(NT) void k_split(const ull *__restrict__ k,
                                              const int32_t *__restrict__ v, long long n,
                                              int lab_bits, int32_t *__restrict__ perm,
                                              int32_t *__restrict__ lab) {
  const ull mask = (lab_bits >= 64) ? ~0ull : ((1ull << lab_bits) - 1ull);
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    perm[i] = v[i];
    lab[i] = (int32_t)(k[i] & mask);
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

// Claim key k in bitmap bm; true for exactly one caller per key.
__device__ __forceinline__ bool claim(uint32_t *bm, uint32_t k) {
  const uint32_t bit = 1u << (k & 31u);
  uint32_t *w = bm + (k >> 5);
  if (*w & bit) return false;  // already set (a stale zero falls through)
  return (atomicOr(w, bit) & bit) == 0;
}

// Append `key` for every lane with `want`, one atomic per wavefront.
__device__ __forceinline__ void wave_push(bool want, uint32_t key, uint32_t *q, uint32_t cap,
                                          Scalars *sc) {
  unsigned long long m = __ballot(want);
  if (m == 0) return;
  const int leader = __ffsll(m) - 1;
  uint32_t base = 0;
  if ((int)__lane_id() == leader) base = atomicAdd(&sc->tail, (uint32_t)__popcll(m));
  base = __shfl(base, leader, WAVE);
  if (want) {
    uint32_t pos = base + (uint32_t)__popcll(m & __lanemask_lt());
    if (pos < cap) q[pos] = key;
    else atomicOr(&sc->overflow, 1u);
  }
}

// Per-key move structure of a forward key (also used by compaction).
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

__device__ __forceinline__ uint32_t fwd_units(const Problem &P, uint32_t key) {
  Fwd s = fwd_info(P, key);
  return s.eA + (uint32_t)s.be + s.mU;
}

// One forward work unit: an A-epsilon arc, a B-epsilon arc, or one arc of the
// smaller non-epsilon side joined against the other side's label bucket.
__device__ __forceinline__ void fwd_unit(const Problem &P, uint32_t key, uint32_t local,
                                         uint32_t *q, uint32_t cap, Scalars *sc, ull &gen) {
  const Fwd s = fwd_info(P, key);
  const uint32_t sh = P.shiftB;
  if (local < s.eA) {
    int32_t ea = P.aOut.perm[s.aS + (int32_t)local];
    uint32_t d = make_key((uint32_t)P.A.dst[ea], s.qb, 0u, sh);
    ++gen;
    wave_push(claim(P.vis, d), d, q, cap, sc);
  } else if (local < s.eA + (uint32_t)s.be) {
    int32_t eb = P.bOut.perm[s.bS + (int32_t)(local - s.eA)];
    uint32_t d = make_key(s.qa, (uint32_t)P.B.dst[eb], s.ae > 0 ? 1u : 0u, sh);
    ++gen;
    wave_push(claim(P.vis, d), d, q, cap, sc);
  } else {
    const uint32_t j = local - s.eA - (uint32_t)s.be;
    if (s.nA <= s.nB) {
      const int32_t pa = s.aS + s.ae + (int32_t)j;
      const int32_t lab = P.aOut.lab[pa];
      const uint32_t da = (uint32_t)P.A.dst[P.aOut.perm[pa]];
      const int32_t lo = lower_bound_i32(P.bOut.lab, s.bS + s.be, s.bE, lab);
      const int32_t hi = upper_bound_i32(P.bOut.lab, lo, s.bE, lab);
      for (int32_t p = lo; p < hi; ++p) {
        uint32_t d = make_key(da, (uint32_t)P.B.dst[P.bOut.perm[p]], 0u, sh);
        ++gen;
        wave_push(claim(P.vis, d), d, q, cap, sc);
      }
    } else {
      const int32_t pb = s.bS + s.be + (int32_t)j;
      const int32_t lab = P.bOut.lab[pb];
      const uint32_t db = (uint32_t)P.B.dst[P.bOut.perm[pb]];
      const int32_t lo = lower_bound_i32(P.aOut.lab, s.aS + s.ae, s.aE, lab);
      const int32_t hi = upper_bound_i32(P.aOut.lab, lo, s.aE, lab);
      for (int32_t p = lo; p < hi; ++p) {
        uint32_t d = make_key((uint32_t)P.A.dst[P.aOut.perm[p]], db, 0u, sh);
        ++gen;
        wave_push(claim(P.vis, d), d, q, cap, sc);
      }
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

__device__ __forceinline__ uint32_t bwd_units(const Problem &P, uint32_t key) {
  Bwd s = bwd_info(P, key);
  return s.eA + s.eB + s.mU;
}

__device__ __forceinline__ void bwd_try(const Problem &P, uint32_t p, uint32_t *q, uint32_t cap,
                                        Scalars *sc) {
  bool want = test_bit(P.vis, p) && claim(P.coacc, p);
  wave_push(want, p, q, cap, sc);
}

__device__ __forceinline__ void bwd_unit(const Problem &P, uint32_t key, uint32_t local,
                                         uint32_t *q, uint32_t cap, Scalars *sc) {
  const Bwd s = bwd_info(P, key);
  const uint32_t sh = P.shiftB;
  if (local < s.eA) {
    int32_t ea = P.aIn.perm[s.aS + (int32_t)local];
    bwd_try(P, make_key((uint32_t)P.A.src[ea], s.vb, 0u, sh), q, cap, sc);
  } else if (local < s.eA + s.eB) {
    int32_t eb = P.bIn.perm[s.bS + (int32_t)(local - s.eA)];
    uint32_t ub = (uint32_t)P.B.src[eb];
    bwd_try(P, make_key(s.va, ub, 0u, sh), q, cap, sc);
    if (s.epsV) bwd_try(P, make_key(s.va, ub, 1u, sh), q, cap, sc);
  } else {
    const uint32_t j = local - s.eA - s.eB;
    if (s.nA <= s.nB) {
      const int32_t pa = s.aS + s.ae + (int32_t)j;
      const int32_t lab = P.aIn.lab[pa];
      const uint32_t ua = (uint32_t)P.A.src[P.aIn.perm[pa]];
      const bool fa = P.aOut.neps[ua] > 0;
      const int32_t lo = lower_bound_i32(P.bIn.lab, s.bS + s.be, s.bE, lab);
      const int32_t hi = upper_bound_i32(P.bIn.lab, lo, s.bE, lab);
      for (int32_t p = lo; p < hi; ++p) {
        uint32_t ub = (uint32_t)P.B.src[P.bIn.perm[p]];
        bwd_try(P, make_key(ua, ub, 0u, sh), q, cap, sc);
        if (fa) bwd_try(P, make_key(ua, ub, 1u, sh), q, cap, sc);
      }
    } else {
      const int32_t pb = s.bS + s.be + (int32_t)j;
      const int32_t lab = P.bIn.lab[pb];
      const uint32_t ub = (uint32_t)P.B.src[P.bIn.perm[pb]];
      const int32_t lo = lower_bound_i32(P.aIn.lab, s.aS + s.ae, s.aE, lab);
      const int32_t hi = upper_bound_i32(P.aIn.lab, lo, s.aE, lab);
      for (int32_t p = lo; p < hi; ++p) {
        uint32_t ua = (uint32_t)P.A.src[P.aIn.perm[p]];
        bwd_try(P, make_key(ua, ub, 0u, sh), q, cap, sc);
        if (P.aOut.neps[ua] > 0) bwd_try(P, make_key(ua, ub, 1u, sh), q, cap, sc);
      }
    }
  }
}

// Level expansion over qin[lo, hi).  Each workgroup takes NT keys, computes
// their work units, scans them in LDS and deals the units to its threads in
// rounds of NT, so a key with thousands of epsilon arcs is split across the
// whole workgroup.
template <bool FWD>
__global__ __launch_bounds__(NT) void k_expand(Problem P, const uint32_t *__restrict__ qin,
                                               uint32_t lo, uint32_t hi, uint32_t *qout,
                                               uint32_t cap, Scalars *sc) {
  __shared__ uint32_t s_key[NT];
  __shared__ ull s_off[NT + 1];
  __shared__ ull s_w[NWAVES];
  ull gen = 0;
  for (ull base = (ull)lo + (ull)blockIdx.x * NT; base < hi; base += (ull)gridDim.x * NT) {
    const ull i = base + threadIdx.x;
    uint32_t key = 0;
    ull units = 0;
    if (i < hi) {
      key = qin[i];
      units = FWD ? fwd_units(P, key) : bwd_units(P, key);
    }
    ull total;
    ull ex = block_excl_scan<ull>(units, s_w, total);
    s_key[threadIdx.x] = key;
    s_off[threadIdx.x] = ex;
    if (threadIdx.x == 0) s_off[NT] = total;
    __syncthreads();
    for (ull r = 0; r < total; r += NT) {
      const ull u = r + threadIdx.x;
      if (u < total) {
        // owner = largest o with s_off[o] <= u (it has units > 0)
        int a = 0, b = NT - 1;
        while (a < b) {
          int mid = (a + b + 1) >> 1;
          if (s_off[mid] <= u) a = mid; else b = mid - 1;
        }
        const uint32_t local = (uint32_t)(u - s_off[a]);
        if (FWD) fwd_unit(P, s_key[a], local, qout, cap, sc, gen);
        else bwd_unit(P, s_key[a], local, qout, cap, sc);
      }
    }
    __syncthreads();
  }
  if (FWD) {
    gen = wave_sum(gen);
    if (__lane_id() == 0 && gen) atomicAdd(&sc->generated, gen);
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

// Start keys (sa, sb, 0) for every pair of start states (Algorithm 1).
__global__ __launch_bounds__(NT) void k_seed(Problem P, const int32_t *__restrict__ la,
                                             const uint32_t *__restrict__ na_p,
                                             const int32_t *__restrict__ lb,
                                             const uint32_t *__restrict__ nb_p, uint32_t *q,
                                             uint32_t cap, Scalars *sc) {
  const ull na = *na_p, nb = *nb_p, n = na * nb;
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    bool want = false;
    uint32_t k = 0;
    if (i < n) {
      k = make_key((uint32_t)la[i / nb], (uint32_t)lb[i % nb], 0u, P.shiftB);
      want = claim(P.vis, k);
    }
    wave_push(want, k, q, cap, sc);
  }
}

__global__ __launch_bounds__(NT) void k_bwd_seed(Problem P, const uint32_t *__restrict__ fq,
                                                 uint32_t n, uint32_t *bq, uint32_t cap,
                                                 Scalars *sc) {
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    bool want = false;
    uint32_t k = 0;
    if (i < n) {
      k = fq[i];
      uint32_t qa = key_qa(k, P.shiftB), qb = key_qb(k, P.shiftB);
      if (P.A.accept[qa] && P.B.accept[qb]) want = claim(P.coacc, k);
    }
    wave_push(want, k, bq, cap, sc);
  }
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
// the label groups of the side with fewer non-epsilon arcs and binary-searches
// the other side's bucket; each group is emitted row-major (a outer, b inner).
template <class Visit>
__device__ __forceinline__ void enum_light(const Problem &P, const Fwd &s, Visit &&vis) {
  const uint32_t sh = P.shiftB;
  for (int32_t p = s.aS; p < s.aS + (int32_t)s.eA; ++p) {
    int32_t ea = P.aOut.perm[p];
    vis(make_key((uint32_t)P.A.dst[ea], s.qb, 0u, sh), P.A.il[ea], 0, P.A.w[ea], ea, -1);
  }
  const uint32_t f2 = s.ae > 0 ? 1u : 0u;
  for (int32_t p = s.bS; p < s.bS + s.be; ++p) {
    int32_t eb = P.bOut.perm[p];
    vis(make_key(s.qa, (uint32_t)P.B.dst[eb], f2, sh), 0, P.B.ol[eb], P.B.w[eb], -1, eb);
  }
  if (!s.mU) return;
  if (s.nA <= s.nB) {
    int32_t p = s.aS + s.ae, bl = s.bS + s.be;
    while (p < s.aE) {
      const int32_t lab = P.aOut.lab[p];
      int32_t pend = p + 1;
      while (pend < s.aE && P.aOut.lab[pend] == lab) ++pend;
      const int32_t lo = lower_bound_i32(P.bOut.lab, bl, s.bE, lab);
      const int32_t hi = upper_bound_i32(P.bOut.lab, lo, s.bE, lab);
      bl = hi;
      for (int32_t pa = p; pa < pend && lo < hi; ++pa) {
        const int32_t ea = P.aOut.perm[pa];
        const uint32_t da = (uint32_t)P.A.dst[ea];
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        for (int32_t pb = lo; pb < hi; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          vis(make_key(da, (uint32_t)P.B.dst[eb], 0u, sh), ia, P.B.ol[eb], wa + P.B.w[eb], ea, eb);
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
      const int32_t lo = lower_bound_i32(P.aOut.lab, al, s.aE, lab);
      const int32_t hi = upper_bound_i32(P.aOut.lab, lo, s.aE, lab);
      al = hi;
      for (int32_t pa = lo; pa < hi; ++pa) {
        const int32_t ea = P.aOut.perm[pa];
        const uint32_t da = (uint32_t)P.A.dst[ea];
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        for (int32_t pb = p; pb < pend; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          vis(make_key(da, (uint32_t)P.B.dst[eb], 0u, sh), ia, P.B.ol[eb], wa + P.B.w[eb], ea, eb);
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
      d = make_key((uint32_t)P.A.dst[ea], s.qb, 0u, sh);
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
      d = make_key(s.qa, (uint32_t)P.B.dst[eb], f2, sh);
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
      uint32_t kept = 0;
      if (i < s.nA) {
        const int32_t pa = s.aS + s.ae + (int32_t)i;
        const int32_t lab = P.aOut.lab[pa];
        ea = P.aOut.perm[pa];
        lo = lower_bound_i32(P.bOut.lab, s.bS + s.be, s.bE, lab);
        hi = upper_bound_i32(P.bOut.lab, lo, s.bE, lab);
        const uint32_t da = (uint32_t)P.A.dst[ea];
        for (int32_t pb = lo; pb < hi; ++pb)
          kept += test_bit(P.coacc, make_key(da, (uint32_t)P.B.dst[P.bOut.perm[pb]], 0u, sh));
      }
      uint32_t tot;
      uint32_t ex = block_excl_scan<uint32_t>(kept, s_w, tot);
      if (FILL && kept) {
        const uint32_t da = (uint32_t)P.A.dst[ea];
        const int32_t ia = P.A.il[ea];
        const float wa = P.A.w[ea];
        uint32_t pos = pos0 + run + ex;
        for (int32_t pb = lo; pb < hi; ++pb) {
          const int32_t eb = P.bOut.perm[pb];
          const uint32_t d = make_key(da, (uint32_t)P.B.dst[eb], 0u, sh);
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

hipError_t build_view(const DevGraph &g, int side, bool by_dst, int lab_bits, int32_t *perm,
                      int32_t *lab, int32_t *neps, int32_t *off_out, unsigned long long *k0,
                      int32_t *v0, unsigned long long *k1, int32_t *v1, void *sort_temp,
                      uint32_t *eps_states, hipStream_t s) {
  const size_t E = (size_t)g.E;
  hipError_t e;
  if (E) {
    k_make_keys<<<grid_for(E), NT, 0, s>>>(g, side, by_dst ? 1 : 0, lab_bits, k0, v0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int bits = bitlen((unsigned long long)(g.V > 0 ? g.V - 1 : 0)) + lab_bits;
    if ((e = radix_sort(k0, v0, k1, v1, E, bits, sort_temp, s)) != hipSuccess) return e;
    k_split<<<grid_for(E), NT, 0, s>>>(k0, v0, (long long)E, lab_bits, perm, lab);
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
  }
  return hipSuccess;
}

hipError_t launch_seed_lists(const Problem &P, int32_t *la, uint32_t *na, int32_t *lb,
                             uint32_t *nb, uint32_t *queue, uint32_t cap, Scalars *sc,
                             hipStream_t s) {
  k_collect<<<grid_for((size_t)P.A.V, 1024), NT, 0, s>>>(P.A.start, P.A.V, la, na);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_collect<<<grid_for((size_t)P.B.V, 1024), NT, 0, s>>>(P.B.start, P.B.V, lb, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_seed<<<64, NT, 0, s>>>(P, la, na, lb, nb, queue, cap, sc);
  return hipGetLastError();
}

hipError_t launch_expand(const Problem &P, bool forward, const uint32_t *qin, uint32_t lo,
                         uint32_t hi, uint32_t *qout, uint32_t cap, Scalars *sc,
                         hipStream_t s) {
  if (hi <= lo) return hipSuccess;
  unsigned g = grid_for((size_t)(hi - lo), 8192);
  if (forward) k_expand<true><<<g, NT, 0, s>>>(P, qin, lo, hi, qout, cap, sc);
  else k_expand<false><<<g, NT, 0, s>>>(P, qin, lo, hi, qout, cap, sc);
  return hipGetLastError();
}

hipError_t launch_bwd_seed(const Problem &P, const uint32_t *fq, uint32_t n, uint32_t *bq,
                           uint32_t cap, Scalars *sc, hipStream_t s) {
  if (!n) return hipSuccess;
  k_bwd_seed<<<grid_for(n, 8192), NT, 0, s>>>(P, fq, n, bq, cap, sc);
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
