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
// Validation also notes whether some state's arcs are not ordered by the
// matched label (then the out-view is sorted; otherwise it is the input).
constexpr uint32_t INFO_UNSORTED = 1u << 16;

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

// The state id in an arc record's neighbour field.
__device__ __forceinline__ uint32_t nbr_of(int32_t y) { return (uint32_t)(y & NBR_MASK); }

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
// VAL_ITEMS items per thread and round: the loads of all of them are issued
// before any check (the source check's offsets depend on the source).
constexpr int VAL_ITEMS = 8;

__global__ __launch_bounds__(NT) void k_validate(DevGraph g, int side, uint32_t *err,
                                                 uint32_t *maxlab, uint32_t *nacc) {
  uint32_t bits = 0, mx = 0, na = 0;
  const long long V = g.V, E = g.E;
  const long long n = (V + 1 > E) ? V + 1 : E;
  const long long tile = (long long)NT * VAL_ITEMS;
  for (long long base = (long long)blockIdx.x * tile; base < n;
       base += (long long)gridDim.x * tile) {
    // states: offsets and flags
    int32_t oa[VAL_ITEMS], ob[VAL_ITEMS];
    uint8_t st[VAL_ITEMS], ac[VAL_ITEMS];
#pragma unroll
    for (int r = 0; r < VAL_ITEMS; ++r) {
      const long long i = base + (long long)r * NT + threadIdx.x;
      oa[r] = ob[r] = 0;
      st[r] = ac[r] = 0;
      if (i <= V) oa[r] = g.off[i];
      if (i < V) {
        ob[r] = g.off[i + 1];
        st[r] = g.start[i];
        ac[r] = g.accept[i];
      }
    }
    // arcs: source and target, then the source's offsets
    int32_t sr[VAL_ITEMS], ds[VAL_ITEMS], s0[VAL_ITEMS], s1[VAL_ITEMS];
#pragma unroll
    for (int r = 0; r < VAL_ITEMS; ++r) {
      const long long i = base + (long long)r * NT + threadIdx.x;
      sr[r] = -1;
      ds[r] = 0;
      if (i < E) {
        sr[r] = g.src[i];
        ds[r] = g.dst[i];
      }
    }
#pragma unroll
    for (int r = 0; r < VAL_ITEMS; ++r) {
      s0[r] = s1[r] = 0;
      if (sr[r] >= 0 && sr[r] < V) {
        s0[r] = g.off[sr[r]];
        s1[r] = g.off[sr[r] + 1];
      }
    }
#pragma unroll
    for (int r = 0; r < VAL_ITEMS; ++r) {
      const long long i = base + (long long)r * NT + threadIdx.x;
      if (i == 0 && oa[r] != 0) bits |= ERR_OFFSETS;
      if (i == V && oa[r] != E) bits |= ERR_OFFSETS;
      if (i < V) {
        if (ob[r] < oa[r]) bits |= ERR_OFFSETS;
        if (st[r] > 1 || ac[r] > 1) bits |= ERR_FLAG;
        na += ac[r] == 1 ? 1u : 0u;
      }
      if (i < E) {
        const int32_t sv = sr[r], d = ds[r];
        if (d < 0 || d >= V) bits |= ERR_DST;
        const bool src_ok = sv >= 0 && sv < V && s0[r] <= i && i < s1[r];
        if (!src_ok) bits |= ERR_SRC;
        if (side != 2) {
          const int32_t il = g.il[i], ol = g.ol[i];
          if (il < 0 || ol < 0) bits |= ERR_LABEL;
          if (src_ok && i > s0[r] &&
              (side == 0 ? g.ol[i - 1] : g.il[i - 1]) > (side == 0 ? ol : il))
            bits |= INFO_UNSORTED;  // not an error: the out-view needs a sort
          const int32_t lab = side == 0 ? ol : il;
          if (lab > 0 && (uint32_t)lab > mx) mx = (uint32_t)lab;
        }
      }
    }
  }
  // one atomic per workgroup: same-address atomics serialize
  __shared__ uint32_t s_bits[NWAVES], s_mx[NWAVES], s_na[NWAVES];
  bits = wave_or(bits);
  mx = wave_max(mx);
  na = wave_sum(na);
  if (__lane_id() == 0) {
    s_bits[threadIdx.x / WAVE] = bits;
    s_mx[threadIdx.x / WAVE] = mx;
    s_na[threadIdx.x / WAVE] = na;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NWAVES; ++w) {
      bits |= s_bits[w];
      mx = s_mx[w] > mx ? s_mx[w] : mx;
      na += s_na[w];
    }
    if (bits) atomicOr(err, bits);
    if (mx) atomicMax(maxlab, mx);
    if (na && nacc) atomicAdd(nacc, na);
  }
}

// What the composition needs from a graph whose structure the caller
// vouches for (validation switched off): the largest matched label, whether
// the arcs of every state are in label order (an arc and the one before it
// with the same source), and the number of accepting states; no checks.
__global__ __launch_bounds__(NT) void k_label_facts(DevGraph g, int side, uint32_t *err,
                                                    uint32_t *maxlab, uint32_t *nacc) {
  uint32_t bits = 0, mx = 0, na = 0;
  const long long V = g.V, E = g.E;
  const long long n = V > E ? V : E;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    if (i < V && nacc) na += g.accept[i] == 1 ? 1u : 0u;
    if (i < E && side != 2) {
      const int32_t lab = side == 0 ? g.ol[i] : g.il[i];
      if (lab > 0 && (uint32_t)lab > mx) mx = (uint32_t)lab;
      if (i > 0 && g.src[i - 1] == g.src[i] && (side == 0 ? g.ol[i - 1] : g.il[i - 1]) > lab)
        bits |= INFO_UNSORTED;
    }
  }
  __shared__ uint32_t s_bits[NWAVES], s_mx[NWAVES], s_na[NWAVES];
  bits = wave_or(bits);
  mx = wave_max(mx);
  na = wave_sum(na);
  if (__lane_id() == 0) {
    s_bits[threadIdx.x / WAVE] = bits;
    s_mx[threadIdx.x / WAVE] = mx;
    s_na[threadIdx.x / WAVE] = na;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < NWAVES; ++w) {
      bits |= s_bits[w];
      mx = s_mx[w] > mx ? s_mx[w] : mx;
      na += s_na[w];
    }
    if (bits) atomicOr(err, bits);
    if (mx) atomicMax(maxlab, mx);
    if (na && nacc) atomicAdd(nacc, na);
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
                                              int side, int32_t *__restrict__ perm,
                                              int32_t *__restrict__ olab, float *__restrict__ wv,
                                              int2 *__restrict__ arec) {
  const ull mask = (lab_bits >= 64) ? ~0ull : ((1ull << lab_bits) - 1ull);
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    // without sorted pairs (k null) the arcs are already in view order
    const int32_t e = k ? v[i] : (int32_t)i;
    perm[i] = e;
    if (olab) {
      olab[i] = side == 0 ? g.il[e] : g.ol[e];
      wv[i] = g.w[e];
    }
    int32_t nb = by_dst ? g.src[e] : g.dst[e];
    if (eps_rec && eps_rec[2 * (size_t)nb].y > 0) nb |= NBR_EPS;
    arec[i] = make_int2(k ? (int32_t)(k[i] & mask) : (side == 0 ? g.ol[e] : g.il[e]), nb);
  }
}

// off[v] = first sorted position whose group is >= v (v = 0..V).
// off[v] = first position whose key's group is >= v, for v <= V: by binary
// search (one thread per group; for graphs with few arcs per state) ...
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

// ... or from adjacent keys (one thread per position; runs of empty groups
// are short when there are at least a few arcs per four states)
__global__ __launch_bounds__(NT) void k_group_bounds(const ull *__restrict__ k, long long n,
                                                     int V, int lab_bits,
                                                     int32_t *__restrict__ off) {
  // position i (0 <= i <= n) starts the groups after the group of key i - 1
  // up to the group of key i (groups past the last key start at n)
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i <= n;
       i += (long long)gridDim.x * NT) {
    const long long g0 = i > 0 ? (long long)(k[i - 1] >> lab_bits) + 1 : 0;
    const long long g1 = i < n ? (long long)(k[i] >> lab_bits) : (long long)V;
    for (long long v = g0; v <= g1; ++v) off[v] = (int32_t)i;
  }
}

// State records.  eps_mode: 0 = no epsOutA flag (views of B), 1 = A's
// out-view (flag from its own epsilon count), 2 = A's in-view (flag from
// A's out-view records in eps_rec).
__global__ __launch_bounds__(NT) void k_state_rec(const int32_t *__restrict__ off,
                                                  const int2 *__restrict__ arec, int V,
                                                  const uint8_t *__restrict__ accept,
                                                  const uint8_t *__restrict__ start,
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
    if ((eps_mode == 1 && n > 0) || (eps_mode == 2 && eps_rec[2 * v].y > 0))
      flags |= (int32_t)FLAG_EPS_OUT;
    if (start && start[v]) flags |= (int32_t)FLAG_START;
    srec[2 * v] = make_int4(s0, n, s1, flags);
    neps_states += n > 0 ? 1u : 0u;
  }
  if (eps_states) {
    const uint32_t tot = block_sum(neps_states, s_w);
    if (threadIdx.x == 0 && tot) atomicAdd(eps_states, tot);
  }
}

// Groups longer than this are never marked FLAG_UNIQ in A (their labels are
// not checked one by one).
constexpr int32_t UNIQ_SCAN_MAX = 256;

// The four views are finished together: each kernel runs over the
// concatenated states (or arcs, or bucket entries) of all views; a thread
// finds its view with a few comparisons against the prefix sums.
__device__ __forceinline__ int job_of(const ViewJobs &J, const long long *begin, long long i) {
  int j = 0;
#pragma unroll
  for (int t = 1; t < 4; ++t)
    if (i >= begin[t]) j = t;
  return j;
}

// FLAG_UNIQ of a view's records, from the opposite view's groups.
__global__ __launch_bounds__(NT) void k_mark_unique(ViewJobs J) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < J.vbegin[4];
       i += (long long)gridDim.x * NT) {
    const int j = job_of(J, J.vbegin, i);
    const ViewJob &b = J.j[j];
    const long long v = i - J.vbegin[j];
    const int4 o = b.other[2 * v];
    const int4 me = b.srec[2 * v];
    const int32_t n = o.z - o.x;
    bool u = b.excl[v] == 0;
    if (b.side == 1) {
      u = u && n == 1;
    } else {
      // no epsilon arc of v itself in this view (out-view: no epsilon
      // output; in-view: no epsilon in-arc)
      if (me.y != 0) u = false;
      if (o.y != 0 || n > UNIQ_SCAN_MAX) u = false;
      // eight arcs per round, loaded together
      int32_t last = -1;  // label of the arc before the round (none: -1, labels are >= 0)
      for (int32_t k0 = o.x; u && k0 < o.z; k0 += 8) {
        int2 a[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) a[q] = k0 + q < o.z ? b.other_arec[k0 + q] : make_int2(-1, 0);
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (k0 + q < o.z) {
            if (a[q].y & NBR_EPS) u = false;                       // source has epsilon output
            if ((q ? a[q - 1].x : last) == a[q].x) u = false;      // repeated label
          }
        last = a[7].x;
      }
    }
    if (u) b.srec[2 * v] = make_int4(me.x, me.y, me.z, me.w | (int32_t)FLAG_UNIQ);
  }
}

// Mark every arc whose other end has FLAG_UNIQ in its view.
__global__ __launch_bounds__(NT) void k_mark_arcs(ViewJobs J) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < J.ebegin[4];
       i += (long long)gridDim.x * NT) {
    const int j = job_of(J, J.ebegin, i);
    const ViewJob &b = J.j[j];
    const long long e = i - J.ebegin[j];
    const int2 a = b.arec[e];
    if (b.srec[2 * (size_t)(a.y & NBR_MASK)].w & (int32_t)FLAG_UNIQ)
      b.arec[e] = make_int2(a.x, a.y | NBR_UNIQ);
  }
}

// Second state record: the first epsilon and first non-epsilon arcs; and
// FLAG_DISTINCT in the first.
__global__ __launch_bounds__(NT) void k_state_inline(ViewJobs J) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < J.vbegin[4];
       i += (long long)gridDim.x * NT) {
    const int j = job_of(J, J.vbegin, i);
    const ViewJob &b = J.j[j];
    const long long v = i - J.vbegin[j];
    const int4 r = b.srec[2 * v];
    const int2 first_ne = r.x + r.y < r.z ? b.arec[r.x + r.y] : make_int2(0, 0);
    b.srec[2 * v + 1] = make_int4(r.y > 0 ? b.arec[r.x].y : 0, first_ne.x, first_ne.y, 0);
    // labels are sorted inside the group: distinct unless two neighbours are
    // equal (eight arcs per round, loaded together)
    bool d = r.z - r.x - r.y <= DISTINCT_SCAN_MAX;
    int32_t last = -1;  // label before the round (none: -1, labels are >= 0)
    for (int32_t k0 = r.x + r.y; d && k0 < r.z; k0 += 8) {
      int32_t l[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) l[q] = k0 + q < r.z ? b.arec[k0 + q].x : -1 - q;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if ((q ? l[q - 1] : last) == l[q]) d = false;
      last = l[7];
    }
    if (d) b.srec[2 * v] = make_int4(r.x, r.y, r.z, r.w | (int32_t)FLAG_DISTINCT);
  }
}

// Chain records of the views that have them (see View).
__global__ __launch_bounds__(NT) void k_chains(ViewJobs J) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < J.vbegin[4];
       i += (long long)gridDim.x * NT) {
    const int j = job_of(J, J.vbegin, i);
    const ViewJob &b = J.j[j];
    if (!b.chain) continue;
    const long long v = i - J.vbegin[j];
    int32_t w[4 * CHAIN_INT4] = {};
    int n = 0;
    uint32_t cur = (uint32_t)v;
#pragma unroll
    for (int k = 0; k < CHAIN_STEPS; ++k) {
      if (n == k) {
        const int4 r = b.srec[2 * (size_t)cur];
        const int2 a = r.z - r.x == 1 ? b.arec[r.x] : make_int2(0, 0);
        const bool step = r.z - r.x == 1 && a.x != 0 && (a.y & NBR_UNIQ) &&
                          !(b.out_view && (r.w & (int32_t)FLAG_ACCEPT));
        if (step) {
          w[1 + 2 * k] = a.x;
          w[2 + 2 * k] = a.y;
          cur = (uint32_t)(a.y & NBR_MASK);
          n = k + 1;
        }
      }
    }
    w[0] = n;
    int4 *c = b.chain + CHAIN_INT4 * v;
#pragma unroll
    for (int q = 0; q < CHAIN_INT4; ++q)
      c[q] = make_int4(w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]);
  }
}

// Label buckets: lut[v * S + l] = {first position of label l, first > l,
// neighbour of the first arc (or -1), 0}, for the views that have them.
__global__ __launch_bounds__(NT) void k_build_lut(ViewJobs J) {
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < J.lbegin[4];
       i += (long long)gridDim.x * NT) {
    const int j = job_of(J, J.lbegin, i);
    const ViewJob &b = J.j[j];
    const long long x = i - J.lbegin[j];
    const int32_t v = (int32_t)(x / b.lstride), l = (int32_t)(x % b.lstride);
    const int4 r = b.srec[2 * (size_t)v];
    const int32_t lo = lb_label(b.arec, r.x, r.z, l);
    const int32_t hi = lb_label(b.arec, lo, r.z, l + 1);
    b.lut[x] = make_int4(lo, hi, lo < hi ? b.arec[lo].y : -1, 0);
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

// An opaque copy of a register value.  Selecting between it and a loaded
// value stays a register select: without it the compiler may turn the
// select into a load through a selected pointer, parking the register value
// in scratch memory.
__device__ __forceinline__ int32_t opaque(int32_t x) {
  asm("" : "+v"(x));
  return x;
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

// A state's two records in one view (see View).
struct Rec {
  int4 r0, r1;
};

// An opaque copy of a record pair held in registers (see opaque(int32_t)).
__device__ __forceinline__ Rec opaque(const Rec &r) {
  Rec o;
  o.r0 = make_int4(opaque(r.r0.x), opaque(r.r0.y), opaque(r.r0.z), opaque(r.r0.w));
  o.r1 = make_int4(opaque(r.r1.x), opaque(r.r1.y), opaque(r.r1.z), opaque(r.r1.w));
  return o;
}

__device__ __forceinline__ Rec load_rec(const View &v, uint32_t q) {
  Rec r;
  r.r0 = v.srec[2 * (size_t)q];
  r.r1 = v.srec[2 * (size_t)q + 1];
  return r;
}

// Move structure of a key in the forward direction (also used to write C).
// flA/flB: record flags of qa / qb; e0A/e0B: other end of the first epsilon
// arc of qa / qb; l1, n1: label and other end of the first non-epsilon arc
// (valid when the arc exists).
struct Fwd {
  uint32_t qa, qb, f;
  int32_t aS, ae, aE, bS, be, bE;
  int32_t flA, flB;
  uint32_t eA, nA, nB, mU;
  uint32_t epsA;      // epsOutA(qa)
  uint32_t accept;    // accept(qa) and accept(qb)
  uint32_t uqA, uqB;  // FLAG_UNIQ of qa, qb (out-views)
  uint32_t start;     // a start key: f = 0, start(qa) and start(qb)
  int32_t e0A, e0B, l1A, n1A, l1B, n1B;
};

__device__ __forceinline__ Fwd make_fwd(uint32_t key, uint32_t shiftB, const Rec &A, const Rec &B) {
  Fwd s;
  s.f = key_f(key);
  s.qb = key_qb(key, shiftB);
  s.qa = key_qa(key, shiftB);
  s.aS = A.r0.x;
  s.ae = A.r0.y;
  s.aE = A.r0.z;
  s.flA = A.r0.w;
  s.bS = B.r0.x;
  s.be = B.r0.y;
  s.bE = B.r0.z;
  s.flB = B.r0.w;
  s.e0A = A.r1.x;
  s.l1A = A.r1.y;
  s.n1A = A.r1.z;
  s.e0B = B.r1.x;
  s.l1B = B.r1.y;
  s.n1B = B.r1.z;
  s.epsA = s.ae > 0 ? 1u : 0u;
  s.accept = (uint32_t)(s.flA & s.flB) & FLAG_ACCEPT;
  s.uqA = (uint32_t)s.flA & FLAG_UNIQ;
  s.uqB = (uint32_t)s.flB & FLAG_UNIQ;
  s.start = (s.f == 0 && (s.flA & s.flB & (int32_t)FLAG_START)) ? 1u : 0u;
  s.eA = s.f ? 0u : (uint32_t)s.ae;
  s.nA = (uint32_t)(s.aE - s.aS - s.ae);
  s.nB = (uint32_t)(s.bE - s.bS - s.be);
  s.mU = (s.nA && s.nB) ? (s.nA < s.nB ? s.nA : s.nB) : 0u;
  return s;
}

// The records a move structure was made from.
__device__ __forceinline__ Rec rec_a(const Fwd &s) {
  return Rec{make_int4(s.aS, s.ae, s.aE, s.flA), make_int4(s.e0A, s.l1A, s.n1A, 0)};
}
__device__ __forceinline__ Rec rec_b(const Fwd &s) {
  return Rec{make_int4(s.bS, s.be, s.bE, s.flB), make_int4(s.e0B, s.l1B, s.n1B, 0)};
}

// INL: also load the second records (the inline first arcs); the general
// enumeration of the output passes walks the arc records instead.
template <bool INL = true>
__device__ __forceinline__ Fwd fwd_info(const Problem &P, uint32_t key) {
  const uint32_t qa = key_qa(key, P.shiftB), qb = key_qb(key, P.shiftB);
  Rec A, B;
  if (INL) {
    A = load_rec(P.aOut, qa);
    B = load_rec(P.bOut, qb);
  } else {
    A.r0 = P.aOut.srec[2 * (size_t)qa];
    B.r0 = P.bOut.srec[2 * (size_t)qb];
    A.r1 = B.r1 = make_int4(0, 0, 0, 0);
  }
  return make_fwd(key, P.shiftB, A, B);
}

// Work units of a key: its A-epsilon arcs, its B-epsilon arcs, and the
// non-epsilon arcs of the smaller side (each joined with the other side's
// bucket of its label).
__device__ __forceinline__ uint32_t fwd_units(const Fwd &s) { return s.eA + (uint32_t)s.be + s.mU; }

// The keys a work unit reaches: for p in [lo, hi), with nb_p the neighbour
// field of arc record p (nb_lo given) of the side named by VARY_A (A's view
// when set, else B's), the key whose state on that side is nb_p and whose
// state on the other side is `fixed`, with records `fix` (loaded before the
// bucket lookup resolves, or the current key's own records for epsilon
// moves, so visiting a key loads only the varying side's records).  Forward
// keys take filter bit F_ONE; backward keys are also visited with f = 1 under
// DUAL or, with DUAL_FROM_NB, when NBR_EPS of nb_p (epsOutA of an A-side
// neighbour) is set.  HOT marks keys many threads may reach at once.  A key
// is reached at most once by the search (needs no claim) when FIXED_UNIQ is
// set and nb_p has NBR_UNIQ: both of its states are marked FLAG_UNIQ.
enum : uint32_t { VARY_A = 1, DUAL = 2, DUAL_FROM_NB = 4, HOT = 8, F_ONE = 16, FIXED_UNIQ = 32 };
struct UnitRange {
  int32_t lo, hi, nb0;
  uint32_t fixed, flags;
  Rec fix;
};

__device__ __forceinline__ UnitRange fwd_range(const Problem &P, const Fwd &s, uint32_t u) {
  UnitRange r;
  if (u < s.eA) {  // A-epsilon move
    r.lo = s.aS + (int32_t)u;
    r.hi = r.lo + 1;
    r.fixed = s.qb;
    r.fix = rec_b(s);
    r.flags = VARY_A | HOT | (s.uqB ? FIXED_UNIQ : 0u);
    r.nb0 = u == 0 ? opaque(s.e0A) : P.aOut.arec[r.lo].y;
  } else if (u < s.eA + (uint32_t)s.be) {  // B-epsilon move
    const uint32_t j = u - s.eA;
    r.lo = s.bS + (int32_t)j;
    r.hi = r.lo + 1;
    r.fixed = s.qa;
    r.fix = rec_a(s);
    r.flags = HOT | (s.epsA ? F_ONE : 0u) | (s.uqA ? FIXED_UNIQ : 0u);
    r.nb0 = j == 0 ? opaque(s.e0B) : P.bOut.arec[r.lo].y;
  } else {  // matching moves of one arc of the smaller side
    const uint32_t j = u - s.eA - (uint32_t)s.be;
    if (s.nA <= s.nB) {
      const int2 ar = j == 0 ? make_int2(opaque(s.l1A), opaque(s.n1A))
                             : P.aOut.arec[s.aS + s.ae + (int32_t)j];
      r.fixed = nbr_of(ar.y);
      r.fix = load_rec(P.aOut, r.fixed);
      label_range(P.bOut, s.qb, s.bS + s.be, s.bE, ar.x, r.lo, r.hi, r.nb0);
      r.flags = (ar.y & NBR_UNIQ) ? FIXED_UNIQ : 0u;
    } else {
      const int2 br = j == 0 ? make_int2(opaque(s.l1B), opaque(s.n1B))
                             : P.bOut.arec[s.bS + s.be + (int32_t)j];
      r.fixed = nbr_of(br.y);
      r.fix = load_rec(P.bOut, r.fixed);
      label_range(P.aOut, s.qa, s.aS + s.ae, s.aE, br.x, r.lo, r.hi, r.nb0);
      r.flags = VARY_A | ((br.y & NBR_UNIQ) ? FIXED_UNIQ : 0u);
    }
  }
  return r;
}

// Backward structure of key v = (va, vb, g): the predecessors are the exact
// inverse of the three forward moves.
struct Bwd {
  uint32_t va, vb, g, epsV;
  int32_t aS, ae, aE, bS, be, bE;
  int32_t flA, flB;
  uint32_t eA, eB, nA, nB, mU;
  uint32_t uqA, uqB;  // FLAG_UNIQ of va, vb (in-views)
  int32_t e0A, e0B, l1A, n1A, l1B, n1B;  // inline first arcs, as in Fwd
};

__device__ __forceinline__ Bwd make_bwd(uint32_t key, uint32_t shiftB, const Rec &A, const Rec &B) {
  Bwd s;
  s.g = key_f(key);
  s.vb = key_qb(key, shiftB);
  s.va = key_qa(key, shiftB);
  s.aS = A.r0.x;
  s.ae = A.r0.y;
  s.aE = A.r0.z;
  s.flA = A.r0.w;
  s.bS = B.r0.x;
  s.be = B.r0.y;
  s.bE = B.r0.z;
  s.flB = B.r0.w;
  s.e0A = A.r1.x;
  s.l1A = A.r1.y;
  s.n1A = A.r1.z;
  s.e0B = B.r1.x;
  s.l1B = B.r1.y;
  s.n1B = B.r1.z;
  s.epsV = (s.flA & (int32_t)FLAG_EPS_OUT) ? 1u : 0u;
  s.uqA = (uint32_t)s.flA & FLAG_UNIQ;
  s.uqB = (uint32_t)s.flB & FLAG_UNIQ;
  s.eA = (s.g == 0) ? (uint32_t)s.ae : 0u;       // A-epsilon moves land on f = 0
  s.eB = (s.g == s.epsV) ? (uint32_t)s.be : 0u;  // B-epsilon moves land on f = epsOutA
  s.nA = (uint32_t)(s.aE - s.aS - s.ae);
  s.nB = (uint32_t)(s.bE - s.bS - s.be);
  s.mU = (s.g == 0 && s.nA && s.nB) ? (s.nA < s.nB ? s.nA : s.nB) : 0u;
  return s;
}

__device__ __forceinline__ Rec rec_a(const Bwd &s) {
  return Rec{make_int4(s.aS, s.ae, s.aE, s.flA), make_int4(s.e0A, s.l1A, s.n1A, 0)};
}
__device__ __forceinline__ Rec rec_b(const Bwd &s) {
  return Rec{make_int4(s.bS, s.be, s.bE, s.flB), make_int4(s.e0B, s.l1B, s.n1B, 0)};
}

__device__ __forceinline__ Bwd bwd_info(const Problem &P, uint32_t key) {
  return make_bwd(key, P.shiftB, load_rec(P.aIn, key_qa(key, P.shiftB)),
                  load_rec(P.bIn, key_qb(key, P.shiftB)));
}

__device__ __forceinline__ uint32_t bwd_units(const Bwd &s) { return s.eA + s.eB + s.mU; }

__device__ __forceinline__ UnitRange bwd_range(const Problem &P, const Bwd &s, uint32_t u) {
  UnitRange r;
  if (u < s.eA) {  // predecessor by an A-epsilon move: (ua, vb, 0)
    r.lo = s.aS + (int32_t)u;
    r.hi = r.lo + 1;
    r.fixed = s.vb;
    r.fix = rec_b(s);
    r.flags = VARY_A | HOT | (s.uqB ? FIXED_UNIQ : 0u);
    r.nb0 = u == 0 ? opaque(s.e0A) : P.aIn.arec[r.lo].y;
  } else if (u < s.eA + s.eB) {  // by a B-epsilon move: (va, ub, 0 and 1)
    const uint32_t j = u - s.eA;
    r.lo = s.bS + (int32_t)j;
    r.hi = r.lo + 1;
    r.fixed = s.va;
    r.fix = rec_a(s);
    r.flags = HOT | (s.epsV ? DUAL : 0u) | (s.uqA ? FIXED_UNIQ : 0u);
    r.nb0 = j == 0 ? opaque(s.e0B) : P.bIn.arec[r.lo].y;
  } else {  // by matching moves: (ua, ub, 0 and, if epsOutA(ua), 1)
    const uint32_t j = u - s.eA - s.eB;
    if (s.nA <= s.nB) {
      const int2 ar = j == 0 ? make_int2(opaque(s.l1A), opaque(s.n1A))
                             : P.aIn.arec[s.aS + s.ae + (int32_t)j];
      r.fixed = nbr_of(ar.y);
      r.fix = load_rec(P.aIn, r.fixed);
      label_range(P.bIn, s.vb, s.bS + s.be, s.bE, ar.x, r.lo, r.hi, r.nb0);
      r.flags = ((ar.y & NBR_EPS) ? DUAL : 0u) | ((ar.y & NBR_UNIQ) ? FIXED_UNIQ : 0u);
    } else {
      const int2 br = j == 0 ? make_int2(opaque(s.l1B), opaque(s.n1B))
                             : P.bIn.arec[s.bS + s.be + (int32_t)j];
      r.fixed = nbr_of(br.y);
      r.fix = load_rec(P.bIn, r.fixed);
      label_range(P.aIn, s.va, s.aS + s.ae, s.aE, br.x, r.lo, r.hi, r.nb0);
      r.flags = VARY_A | DUAL_FROM_NB | ((br.y & NBR_UNIQ) ? FIXED_UNIQ : 0u);
    }
  }
  return r;
}

// A key reached by a unit: its key, whether it may be hot or is reached
// only once, and the records of its fixed side.
struct Target {
  uint32_t key;
  bool hot, uniq, fixA;
};

// Calls f(target, fix) for every key of a unit range.
template <bool FWD, class F>
__device__ __forceinline__ void for_range(const Problem &P, const UnitRange &r, F &&f) {
  const uint32_t sh = P.shiftB;
  const bool varyA = (r.flags & VARY_A) != 0, hot = (r.flags & HOT) != 0;
  const int2 *arcs = FWD ? (varyA ? P.aOut.arec : P.bOut.arec) : (varyA ? P.aIn.arec : P.bIn.arec);
  for (int32_t p = r.lo; p < r.hi; ++p) {
    const int32_t y = p == r.lo ? r.nb0 : arcs[p].y;
    const uint32_t nb = nbr_of(y);
    const uint32_t qa = varyA ? nb : r.fixed, qb = varyA ? r.fixed : nb;
    Target t;
    t.hot = hot;
    t.uniq = (r.flags & FIXED_UNIQ) && (y & NBR_UNIQ);
    t.fixA = !varyA;
    if (FWD) {
      t.key = make_key(qa, qb, (r.flags & F_ONE) ? 1u : 0u, sh);
      f(t, r.fix);
    } else {
      const uint32_t nf = ((r.flags & DUAL) || ((r.flags & DUAL_FROM_NB) && (y & NBR_EPS))) ? 2u : 1u;
      for (uint32_t ff = 0; ff < nf; ++ff) {
        t.key = make_key(qa, qb, ff, sh);
        f(t, r.fix);
      }
    }
  }
}

// Direction traits: move structure, unit count and unit ranges.
template <bool FWD>
struct Dir;
template <>
struct Dir<true> {
  typedef Fwd Info;
  static __device__ __forceinline__ Fwd info(const Problem &P, uint32_t k) { return fwd_info(P, k); }
  static __device__ __forceinline__ Fwd make(uint32_t k, uint32_t sh, const Rec &A, const Rec &B) {
    return make_fwd(k, sh, A, B);
  }
  static __device__ __forceinline__ const View &viewA(const Problem &P) { return P.aOut; }
  static __device__ __forceinline__ const View &viewB(const Problem &P) { return P.bOut; }
  static __device__ __forceinline__ uint32_t units(const Fwd &s) { return fwd_units(s); }
  static __device__ __forceinline__ UnitRange range(const Problem &P, const Fwd &s, uint32_t u) {
    return fwd_range(P, s, u);
  }
};
template <>
struct Dir<false> {
  typedef Bwd Info;
  static __device__ __forceinline__ Bwd info(const Problem &P, uint32_t k) { return bwd_info(P, k); }
  static __device__ __forceinline__ Bwd make(uint32_t k, uint32_t sh, const Rec &A, const Rec &B) {
    return make_bwd(k, sh, A, B);
  }
  static __device__ __forceinline__ const View &viewA(const Problem &P) { return P.aIn; }
  static __device__ __forceinline__ const View &viewB(const Problem &P) { return P.bIn; }
  static __device__ __forceinline__ uint32_t units(const Bwd &s) { return bwd_units(s); }
  static __device__ __forceinline__ UnitRange range(const Problem &P, const Bwd &s, uint32_t u) {
    return bwd_range(P, s, u);
  }
};

// Calls f(target, fix) for every key of unit `u` of a key with structure s.
template <bool FWD, class F>
__device__ __forceinline__ void for_unit(const Problem &P, const typename Dir<FWD>::Info &s,
                                         uint32_t u, F &&f) {
  for_range<FWD>(P, Dir<FWD>::range(P, s, u), f);
}

// Where the next generation's work goes.
struct NextGen {
  GenSlot *slot;
  uint32_t qbase, hbase;
};

// List a heavy key for the next generation: one packed atomic gives its
// position and the offset of its first unit, consistently.  Its units take
// a multiple of 8 slots of the generation's unit range (the slots past its
// last unit are skipped), so unit u of every heavy key lands on slots
// congruent to u mod 8: see gen_body.
__device__ __forceinline__ void list_heavy(const SearchArgs &S, const NextGen &nx, uint32_t v,
                                           uint32_t units) {
  const ull slots = ((ull)units + 7) & ~7ull;
  const ull old = atomicAdd(&nx.slot->hpack, (slots << 32) | 1ull);
  const ull pos = (ull)nx.hbase + (old & 0xffffffffull);
  if (pos < S.cap && (old >> 32) + slots < (1ull << 32)) {
    S.heavy[pos] = v;
    S.hoff[pos] = (uint32_t)(old >> 32);
  } else {
    atomicOr(&S.sc->overflow, 2u);
  }
}

// The key a search thread expands next (depth-first continuation).
template <bool FWD>
struct Next {
  uint32_t key;
  typename Dir<FWD>::Info info;
};

// Sets bits `m` of word w without reading the word back (no return value is
// waited for).
__device__ __forceinline__ void set_bits(uint32_t *bm, uint32_t w, uint32_t m) {
  __hip_atomic_fetch_or(bm + w, m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void set_bit(uint32_t *bm, uint32_t b) {
  set_bits(bm, b >> 5, 1u << (b & 31u));
}

// A key reached for the first time (`fresh`).  Forward: if it accepts it is
// marked co-accessible and listed as a seed of the backward search.  Then:
// heavy keys go to the next generation's heavy list; a light key becomes this
// thread's next key (depth-first continuation) if it has none yet and the
// depth budget allows, else it joins the next frontier.
template <bool FWD>
__device__ __forceinline__ void place(const Problem &P, const SearchArgs &S, const NextGen &nx,
                                      bool fresh, uint32_t v, const typename Dir<FWD>::Info &vi,
                                      Next<FWD> &nk, int depth) {
  bool push = false, seed = false;
  if (fresh) {
    const uint32_t u = Dir<FWD>::units(vi);
    if constexpr (FWD) {
      seed = P.mark_accept && vi.accept != 0;
      if (seed) set_bit(P.coacc, search_bit(P, v));
    }
    if (u > LIGHT_SEARCH) {
      list_heavy(S, nx, v, u);
    } else if (nk.key == NO_KEY && depth < P.chain_max) {
      nk.key = v;
      nk.info = vi;
    } else {
      push = true;
    }
  }
  if (FWD) wave_push(seed, v, Pusher{S.acc, S.cap, &S.sc->tail2, S.sc});
  wave_push(push, v, Pusher{S.Q + nx.qbase, S.cap - nx.qbase, &nx.slot->qcount, S.sc});
}

// Visit a move target (forward) or a predecessor (backward, where only
// accessible keys are claimed).  The key's state records are loaded first and
// its claim is issued after them, so both round trips overlap.  A key that
// only one move leads to (uniq) is reached exactly once and just has its bit
// set.  Hot keys (epsilon targets, which many threads may reach at once)
// test-load the bitmap before the atomic.  Backward cold claims set the
// co-accessible bit without looking at the accessible bit first; bits set on
// keys that are not accessible are removed after the search (such keys are
// never expanded: fresh needs both bits).
template <bool FWD>
__device__ __forceinline__ void visit(const Problem &P, const SearchArgs &S, const NextGen &nx,
                                      const Target &t, const Rec &fix, Next<FWD> &nk, int depth) {
  const uint32_t v = t.key;
  // one load for every lane: the records of the side that is not fixed
  const Rec L = load_rec(t.fixA ? Dir<FWD>::viewB(P) : Dir<FWD>::viewA(P),
                         t.fixA ? key_qb(v, P.shiftB) : key_qa(v, P.shiftB));
  const Rec F = opaque(fix);
  const typename Dir<FWD>::Info vi =
      Dir<FWD>::make(v, P.shiftB, t.fixA ? F : L, t.fixA ? L : F);
  const uint32_t sb = search_bit(P, v);
  const uint32_t bit = 1u << (sb & 31u), w = sb >> 5;
  bool fresh;
  // a restricted search expands only keys the other search has reached
  const uint32_t *other = FWD ? P.coacc : P.vis;
  uint32_t *mine = FWD ? P.vis : P.coacc;
  const bool restricted = FWD ? P.restrict_fwd != 0 : P.restrict_bwd != 0;
  if (t.uniq) {
    fresh = !restricted || (other[w] & bit) != 0;
    if (fresh) set_bit(mine, sb);
  } else if (t.hot || (FWD && restricted)) {
    const uint32_t wo = restricted ? other[w] : bit, wm = mine[w];  // one round trip
    fresh = (wo & bit) && !(wm & bit) && (atomicOr(mine + w, bit) & bit) == 0;
  } else {
    const uint32_t wo = restricted ? other[w] : bit;
    const uint32_t old = atomicOr(mine + w, bit);
    fresh = (wo & bit) && !(old & bit);
  }
  place<FWD>(P, S, nx, fresh, v, vi, nk, depth);
}

// Chain jumps.  A key whose only move follows the single arc of its B state
// takes up to CHAIN_STEPS hops from the B state's chain record (one load) and
// one bucket lookup in A per hop; every reached key has both states marked
// FLAG_UNIQ (so it needs no claim) and exactly one move, so it is expanded
// on the spot.  Forward, the reached keys get their accessible bits;
// backward, the accessible bits of all reached keys are loaded at once and
// the jump stops before the first key that is not accessible.  The last key
// reached goes to place(); depth advances by the keys expanded.  Returns
// false (nothing done) when the key does not have that shape.
__device__ __forceinline__ uint32_t state_a(const Fwd &s) { return s.qa; }
__device__ __forceinline__ uint32_t state_b(const Fwd &s) { return s.qb; }
__device__ __forceinline__ uint32_t state_a(const Bwd &s) { return s.va; }
__device__ __forceinline__ uint32_t state_b(const Bwd &s) { return s.vb; }
__device__ __forceinline__ bool chain_shape(const Fwd &s) {
  return s.eA == 0 && s.be == 0 && s.nB == 1 && s.nA >= 1;
}
__device__ __forceinline__ bool chain_shape(const Bwd &s) {
  return s.g == 0 && s.eA == 0 && s.eB == 0 && s.nB == 1 && s.nA >= 1;
}

template <bool FWD>
__device__ __forceinline__ bool chain_jump(const Problem &P, const SearchArgs &S, const NextGen &nx,
                                           const typename Dir<FWD>::Info &info, Next<FWD> &nk,
                                           int &depth) {
  const int4 *chain = FWD ? P.bOut.chain : P.bIn.chain;
  const int4 *lut = FWD ? P.aOut.lut : P.aIn.lut;
  const uint32_t stride = (uint32_t)(FWD ? P.aOut.lstride : P.aIn.lstride);
  if (!chain || !lut || !chain_shape(info) || depth >= P.chain_max) return false;
  const int4 *cr = chain + CHAIN_INT4 * (size_t)state_b(info);
  int32_t cw[4 * CHAIN_INT4];
#pragma unroll
  for (int q = 0; q < CHAIN_INT4; ++q) {
    const int4 c = cr[q];
    cw[4 * q] = c.x;
    cw[4 * q + 1] = c.y;
    cw[4 * q + 2] = c.z;
    cw[4 * q + 3] = c.w;
  }
  int n = cw[0];
  if (n > P.chain_max - depth) n = P.chain_max - depth;
  // The A side of hop i is the bucket of label l_i at the A state hop i - 1
  // reached.  Hop 0 is looked up first; the buckets of the later hops are
  // then loaded together at A states guessed to continue with the step hop
  // 0 took (chains of consecutively numbered states take two round trips
  // instead of one per hop).  A hop whose guessed A state differs from the
  // one the previous hop reached ends the jump there; the key it reached is
  // expanded next, which continues the chain.
  const uint32_t VA = (uint32_t)P.A.V;
  uint32_t qa[CHAIN_STEPS];  // A state reached by hop i, for i < done
  int done = 0;
  {
    const uint32_t q0 = state_a(info);
    if (n > 0 && (uint32_t)cw[1] < stride) {
      const int4 b = lut[(size_t)q0 * stride + (uint32_t)cw[1]];
      if (b.y - b.x == 1 && (b.z & NBR_UNIQ) && !(b.z & NBR_EPS)) {
        qa[0] = nbr_of(b.z);
        done = 1;
      }
    }
    if (done == 0) return false;
    const uint32_t step = qa[0] - q0;  // modulo 2^32
    uint32_t nbv[CHAIN_STEPS];  // A state hop i reaches from its guessed state, or NO_KEY
#pragma unroll
    for (int i = 1; i < CHAIN_STEPS; ++i) {
      const uint32_t g = qa[0] + (uint32_t)(i - 1) * step;
      const uint32_t lab = (uint32_t)cw[1 + 2 * i];
      nbv[i] = NO_KEY;
      if (i < n && g < VA && lab < stride) {
        const int4 b = lut[(size_t)g * stride + lab];
        if (b.y - b.x == 1 && (b.z & NBR_UNIQ) && !(b.z & NBR_EPS)) nbv[i] = nbr_of(b.z);
      }
    }
#pragma unroll
    for (int i = 1; i < CHAIN_STEPS; ++i) {
      const uint32_t g = qa[0] + (uint32_t)(i - 1) * step;
      if (i < n && done == i && g == qa[i - 1] && nbv[i] != NO_KEY) {
        qa[i] = nbv[i];
        done = i + 1;
      }
    }
  }
  uint32_t sbs[CHAIN_STEPS];
#pragma unroll
  for (int i = 0; i < CHAIN_STEPS; ++i)
    sbs[i] = i < done ? search_bit(P, make_key(qa[i], nbr_of(cw[2 + 2 * i]), 0u, P.shiftB)) : 0u;
  // a restricted search keeps the reached keys up to the first one the other
  // search has not reached (their bits are loaded together)
  const uint32_t *other = FWD ? P.coacc : P.vis;
  uint32_t *mine = FWD ? P.vis : P.coacc;
  const bool restricted = FWD ? P.restrict_fwd != 0 : P.restrict_bwd != 0;
  bool ok[CHAIN_STEPS];
#pragma unroll
  for (int i = 0; i < CHAIN_STEPS; ++i) ok[i] = i < done && (!restricted || test_bit(other, sbs[i]));
  int m = 0;  // keys reached and kept
#pragma unroll
  for (int i = 0; i < CHAIN_STEPS; ++i)
    if (m == i && ok[i]) m = i + 1;
  // their bits, one atomic per run of keys in the same bitmap word (a chain
  // whose A and B states both advance by one stays on one diagonal)
  uint32_t mw = 0, mm = 0;
#pragma unroll
  for (int i = 0; i < CHAIN_STEPS; ++i)
    if (i < m) {
      if (mm && (sbs[i] >> 5) != mw) {
        set_bits(mine, mw, mm);
        mm = 0;
      }
      mw = sbs[i] >> 5;
      mm |= 1u << (sbs[i] & 31u);
    }
  if (mm) set_bits(mine, mw, mm);
  depth += m > 0 ? m - 1 : 0;
  if (m > 0) {
    uint32_t la = qa[0], lb = (uint32_t)cw[2];
#pragma unroll
    for (int i = 1; i < CHAIN_STEPS; ++i)
      if (i < m) {
        la = qa[i];
        lb = (uint32_t)cw[2 + 2 * i];
      }
    const uint32_t last = make_key(la, nbr_of(lb), 0u, P.shiftB);
    place<FWD>(P, S, nx, true, last, Dir<FWD>::info(P, last), nk, depth);
  }
  return true;
}

// Generation g (one kernel): one thread per unit slot of the generation's
// heavy keys, then one thread per light frontier key.  A thread expands its
// units, then, depth-first, the light keys it reached first (one loop, so
// the visit code exists once).  New work goes to the slot of generation
// g + 1.  Workgroups are dispatched to the eight XCDs in turn (workgroup b
// to XCD b mod 8), and the workgroups of XCD x take the items congruent to
// x mod 8: unit u of a heavy key is expanded on XCD u mod 8, so the keys
// reached from units with the same residue (in a lexicon, the words whose
// entry arcs have it) and the records and bitmap lines they touch stay in
// one XCD's L2.  nb is a multiple of 8.
template <bool FWD>
__device__ __forceinline__ void gen_body(const Problem &P, const SearchArgs &S, int g,
                                         unsigned bid, unsigned nb) {
  typedef typename Dir<FWD>::Info Info;
  Scalars *sc = S.sc;
  const uint32_t ovf = sc->overflow;  // loaded with the slot (one round trip)
  const GenSlot cur = S.G[g % 3];
  const uint32_t hcount = (uint32_t)(cur.hpack & 0xffffffffull);
  const ull U = cur.hpack >> 32;
  // a heavy list of at most NT keys is searched in LDS
  __shared__ uint32_t s_ho[NT], s_hk[NT];
  if (threadIdx.x < hcount) {
    s_ho[threadIdx.x] = S.hoff[cur.hbase + threadIdx.x];
    s_hk[threadIdx.x] = S.heavy[cur.hbase + threadIdx.x];
  }
  __syncthreads();
  if (ovf) return;
  NextGen nx;
  nx.slot = &S.G[(g + 1) % 3];
  nx.qbase = cur.qbase + cur.qcount;
  nx.hbase = cur.hbase + hcount;
  if (bid == 0 && threadIdx.x == 0) {
    nx.slot->qbase = nx.qbase;  // read by generation g + 1 only
    nx.slot->hbase = nx.hbase;
    GenSlot *done = &S.G[(g + 2) % 3];  // generation g - 1: free
    done->qcount = 0;
    done->hpack = 0;
    if (U + cur.qcount) *S.gens = (uint32_t)g + 1;
  }
  const uint32_t *hk = S.heavy + cur.hbase;
  const uint32_t *ho = S.hoff + cur.hbase;
  const ull n = U + cur.qcount;
  const unsigned xcd = bid & 7u, nl = nb >> 3;
  for (ull j = (ull)(bid >> 3) * NT + threadIdx.x; (bid >> 3) < nl; j += (ull)nl * NT) {
    const ull i = 8 * j + xcd;
    if (i >= n) break;
    uint32_t key, u0 = 0, u1 = 0;
    bool one_unit = false;
    if (i < U) {
      uint32_t a = 0, b = hcount - 1;  // largest a with ho[a] <= i
      if (hcount <= NT) {
        while (a < b) {
          const uint32_t mid = (a + b + 1) >> 1;
          if (s_ho[mid] <= i) a = mid; else b = mid - 1;
        }
        key = s_hk[a];
        u0 = (uint32_t)(i - s_ho[a]);
      } else {
        while (a < b) {
          const uint32_t mid = (a + b + 1) >> 1;
          if (ho[mid] <= i) a = mid; else b = mid - 1;
        }
        key = hk[a];
        u0 = (uint32_t)(i - ho[a]);
      }
      one_unit = true;
    } else {
      key = S.Q[cur.qbase + (uint32_t)(i - U)];
    }
    Info info = Dir<FWD>::info(P, key);
    if (one_unit && u0 >= Dir<FWD>::units(info)) continue;  // a slot past the key's units
    u1 = one_unit ? u0 + 1 : Dir<FWD>::units(info);
    for (int depth = 0;; ++depth) {
      Next<FWD> nk;
      nk.key = NO_KEY;
      if (one_unit || !chain_jump<FWD>(P, S, nx, info, nk, depth))
        for (uint32_t u = u0; u < u1; ++u)
          for_unit<FWD>(P, info, u, [&](const Target &t, const Rec &fix) {
            visit<FWD>(P, S, nx, t, fix, nk, depth);
          });
      one_unit = false;
      if (nk.key == NO_KEY) break;
      info = nk.info;
      u0 = 0;
      u1 = Dir<FWD>::units(info);
    }
  }
}

template <bool FWD>
__global__ __launch_bounds__(NT) void k_gen(Problem P, SearchArgs S, int g) {
  gen_body<FWD>(P, S, g, blockIdx.x, gridDim.x);
}

// A forward and a backward search side by side: the first half of the
// workgroups advances the forward search, the second half the backward.
// Held to 128 VGPRs (four wavefronts per SIMD; one more register would
// leave three, and the kernel is bound by the latency of its loads).
__global__ __launch_bounds__(NT, 4) void k_gen2(Problem P, SearchArgs SF, SearchArgs SB, int gf,
                                             int gb) {
  const unsigned half = gridDim.x / 2;
  if (blockIdx.x < half) gen_body<true>(P, SF, gf, blockIdx.x, half);
  else gen_body<false>(P, SB, gb, blockIdx.x - half, half);
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
  const NextGen nx{&S.G[0], 0u, 0u};
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    uint32_t k = 0;
    bool fresh = false;
    Fwd ki;
    if (i < n) {
      k = make_key((uint32_t)la[i / nb], (uint32_t)lb[i % nb], 0u, P.shiftB);
      const uint32_t sb = search_bit(P, k);
      fresh = (!P.restrict_fwd || test_bit(P.coacc, sb)) && claim(P.vis, sb);
      ki = fwd_info(P, k);
    }
    Next<true> nk;
    nk.key = NO_KEY;
    // depth = chain_max: every light start key joins the frontier
    place<true>(P, S, nx, fresh, k, ki, nk, P.chain_max);
  }
}

// Every accepting key (f = 0, and f = 1 where its A state has an epsilon
// output) forms generation 0 of a backward search over all key pairs.
__global__ __launch_bounds__(NT) void k_seed_backward_all(Problem P, SearchArgs S,
                                                          const int32_t *__restrict__ la,
                                                          const uint32_t *__restrict__ na_p,
                                                          const int32_t *__restrict__ lb,
                                                          const uint32_t *__restrict__ nb_p) {
  const ull na = *na_p, nb = *nb_p, n = 2 * na * nb;
  const NextGen nx{&S.G[0], 0u, 0u};
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    uint32_t k = 0;
    bool fresh = false;
    Bwd ki;
    if (i < n) {
      const ull pair = i >> 1;
      const uint32_t qa = (uint32_t)la[pair / nb], f = (uint32_t)(i & 1);
      const bool eps = (P.aOut.srec[2 * (size_t)qa].w & (int32_t)FLAG_EPS_OUT) != 0;
      k = make_key(qa, (uint32_t)lb[pair % nb], f, P.shiftB);
      // every pair is enumerated once, so it is placed once; a forward
      // search running first may already have marked it co-accessible
      fresh = f == 0 || eps;
      if (fresh) set_bit(P.coacc, search_bit(P, k));
      ki = bwd_info(P, k);
    }
    Next<false> nk;
    nk.key = NO_KEY;
    place<false>(P, S, nx, fresh, k, ki, nk, P.chain_max);
  }
}

// The accepting keys listed by the forward search (already co-accessible)
// form generation 0 of the backward search.
__global__ __launch_bounds__(NT) void k_seed_backward(Problem P, SearchArgs S,
                                                      const uint32_t *__restrict__ list) {
  const uint32_t n = S.sc->tail2;
  const NextGen nx{&S.G[0], 0u, 0u};
  for (ull i0 = (ull)blockIdx.x * NT; i0 < n; i0 += (ull)gridDim.x * NT) {
    const ull i = i0 + threadIdx.x;
    const bool valid = i < n;
    const uint32_t k = valid ? list[i] : 0u;
    Bwd ki;
    if (valid) ki = bwd_info(P, k);
    Next<false> nk;
    nk.key = NO_KEY;
    place<false>(P, S, nx, valid, k, ki, nk, P.chain_max);
  }
}

// Number of moves the search examines (a statistic, on request): forward,
// the moves out of the accessible keys (search layout); backward, the
// predecessor moves of the trim keys (key order).
template <bool FWD>
__global__ __launch_bounds__(NT) void k_count_moves(Problem P, ull nwords,
                                                    unsigned long long *__restrict__ out) {
  __shared__ ull s_w[NWAVES];
  const uint32_t *bm = FWD ? P.vis : P.trim;
  ull c = 0;
  const ull nbits = nwords * 32u;
  for (ull k = (ull)blockIdx.x * NT + threadIdx.x; k < nbits; k += (ull)gridDim.x * NT) {
    if (!test_bit(bm, (uint32_t)k)) continue;
    uint32_t key = (uint32_t)k;
    if (FWD) {
      const uint32_t x = (uint32_t)(k >> 1), d = x / P.rowA, qa = x - d * P.rowA;
      key = make_key(qa, (d + qa) & P.maskB, (uint32_t)(k & 1u), P.shiftB);
    }
    const typename Dir<FWD>::Info s = Dir<FWD>::info(P, key);
    const uint32_t nu = Dir<FWD>::units(s);
    for (uint32_t u = 0; u < nu; ++u)
      for_unit<FWD>(P, s, u, [&](const Target &, const Rec &) { ++c; });
  }
  const ull tot = block_sum(c, s_w);
  if (threadIdx.x == 0 && tot) atomicAdd(out, tot);
}

// Number of set bits of a bitmap (one atomic per workgroup).
__global__ __launch_bounds__(NT) void k_popcount(const uint32_t *__restrict__ bm, ull nwords,
                                                 unsigned long long *__restrict__ out) {
  __shared__ ull s_w[NWAVES];
  ull c = 0;
  // four words per load (the bitmaps are 16-byte aligned device buffers)
  const ull n4 = nwords / 4;
  const uint4 *bm4 = reinterpret_cast<const uint4 *>(bm);
#pragma unroll 4
  for (ull w = (ull)blockIdx.x * NT + threadIdx.x; w < n4; w += (ull)gridDim.x * NT) {
    const uint4 q = bm4[w];
    c += (ull)(__popc(q.x) + __popc(q.y) + __popc(q.z) + __popc(q.w));
  }
  for (ull w = 4 * n4 + (ull)blockIdx.x * NT + threadIdx.x; w < nwords;
       w += (ull)gridDim.x * NT)
    c += (ull)__popc(bm[w]);
  const ull tot = block_sum(c, s_w);
  if (threadIdx.x == 0 && tot) atomicAdd(out, tot);
}

// ---------------------------------------------------------------------------
// compaction
// ---------------------------------------------------------------------------

// The trim bitmap in key order: vis AND coacc (which drops co-accessible
// bits of keys that are not accessible), moved from the diagonal search
// layout to rows of one A state (a trim word: 16 B states x 2 f), and
// cnt[w] = popcount(trim[w]).  One tile = TRIM_ROWS A states x TRIM_QB B
// states: the TRIM_QB + TRIM_ROWS - 1 diagonals it meets, TRIM_ROWS / 16
// words of each (the tile's A states), go to LDS; each thread then builds
// four trim words of one A state, 16 diagonals per word.  The workgroups of
// one XCD take consecutive tiles, which share search-bitmap lines.
constexpr uint32_t TRIM_ROWS = 64, TRIM_QB = 256, TRIM_D = TRIM_QB + TRIM_ROWS - 1;

__global__ __launch_bounds__(NT) void k_trim(Problem P, uint32_t VA, uint32_t ntA, ull ntiles,
                                             uint32_t *__restrict__ trim,
                                             uint32_t *__restrict__ cnt) {
  static_assert(NT == 4 * TRIM_ROWS, "four threads per A state of a tile");
  __shared__ uint32_t L[TRIM_D][TRIM_ROWS / 16];
  const uint32_t WR = (P.maskB >> 4) + 1;  // trim words per A state
  const uint32_t rw = P.rowA >> 4;         // search words per diagonal
  const ull first = (ull)(blockIdx.x & 7u) * (gridDim.x >> 3) + (blockIdx.x >> 3);
  const uint32_t r = threadIdx.x >> 2, q = threadIdx.x & 3u;
  for (ull t = first; t < ntiles; t += gridDim.x) {
    const uint32_t a0 = (uint32_t)(t % ntA) * TRIM_ROWS, b0 = (uint32_t)(t / ntA) * TRIM_QB;
    __syncthreads();  // the previous tile's LDS readers are done
    for (uint32_t i = threadIdx.x; i < TRIM_D; i += NT) {
      const uint32_t d = (b0 - a0 - (TRIM_ROWS - 1) + i) & P.maskB;
      const size_t o = (size_t)d * rw + (a0 >> 4);
      const uint4 v = *reinterpret_cast<const uint4 *>(P.vis + o);
      const uint4 c = *reinterpret_cast<const uint4 *>(P.coacc + o);
      L[i][0] = v.x & c.x;
      L[i][1] = v.y & c.y;
      L[i][2] = v.z & c.z;
      L[i][3] = v.w & c.w;
    }
    __syncthreads();
    // trim word j of this A state holds B states b0 + 16 j + [0, 16): key
    // (a0 + r, b0 + 16 j + u) lies on diagonal entry 16 j + u - r + 63
    uint32_t out[4];
#pragma unroll
    for (uint32_t jj = 0; jj < 4; ++jj) {
      const uint32_t j = 4 * q + jj;
      uint32_t wv = 0;
#pragma unroll
      for (uint32_t u = 0; u < 16; ++u)
        wv |= ((L[16 * j + u + (TRIM_ROWS - 1) - r][r >> 4] >> ((r & 15u) * 2)) & 3u) << (2 * u);
      out[jj] = wv;
    }
    const uint32_t qa = a0 + r;
    if (qa < VA) {
      const size_t o = (size_t)qa * WR + (b0 >> 4) + 4 * q;
      if (WR >= 16) {
        *reinterpret_cast<uint4 *>(trim + o) = make_uint4(out[0], out[1], out[2], out[3]);
        *reinterpret_cast<uint4 *>(cnt + o) = make_uint4(__popc(out[0]), __popc(out[1]),
                                                         __popc(out[2]), __popc(out[3]));
      } else {
#pragma unroll
        for (uint32_t jj = 0; jj < 4; ++jj)
          if (4 * q + jj < WR) {
            trim[o + jj] = out[jj];
            cnt[o + jj] = (uint32_t)__popc(out[jj]);
          }
      }
    }
  }
}

// The trim words of output chunk c (trim words [OUT_WORDS c, OUT_WORDS c +
// OUT_WORDS), one per lane): lane l holds its word and the number of keys
// in the chunk's words before it; every lane holds the chunk's key count.  State ids are ranks in key order, so the chunk's
// i-th key is state wbase[first word] + i.
struct TrimChunk {
  uint32_t word, before, count;
  ull w0;  // the chunk's first word
};

__device__ __forceinline__ TrimChunk trim_chunk(const Problem &P, ull chunk, ull nwords) {
  static_assert(OUT_WORDS <= WAVE && (OUT_WORDS & (OUT_WORDS - 1)) == 0,
                "at most one trim word per lane, a power of two");
  TrimChunk t;
  t.w0 = chunk * OUT_WORDS;
  const ull w = t.w0 + __lane_id();
  t.word = __lane_id() < OUT_WORDS && w < nwords ? P.trim[w] : 0u;
  const uint32_t p = (uint32_t)__popc(t.word);
  const uint32_t incl = wave_incl_scan(p);
  t.before = incl - p;
  t.count = __shfl(incl, WAVE - 1, WAVE);
  return t;
}

// The chunk's trim keys in order, as offsets from its first bit (< 2^16),
// in the wavefront's LDS list: each lane writes its word's keys from its
// prefix on.  The list is read by other lanes of the same wavefront only
// (LDS operations of a wavefront complete in order).
__device__ __forceinline__ void trim_expand(const TrimChunk &t, uint16_t *list) {
  static_assert(OUT_WORDS * 32 <= 65536, "offsets fit 16 bits");
  uint32_t m = t.word, o = t.before;
  const uint32_t base = __lane_id() * 32u;
  while (m) {
    list[o++] = (uint16_t)(base + (uint32_t)__ffs(m) - 1u);
    m &= m - 1u;
  }
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ uint32_t trim_key_at(const TrimChunk &t, const uint16_t *list,
                                                uint32_t i) {
  return i < t.count ? (uint32_t)(t.w0 * 32u) + list[i] : 0u;
}

// Kept-arc count of state id: one byte per state; 255 says the count is in
// cnt32 (only such states have an entry there).
__device__ __forceinline__ uint32_t count_of(const uint8_t *__restrict__ cnt8,
                                             const uint32_t *__restrict__ cnt32, ull id) {
  const uint32_t c = cnt8[id];
  return c == 255u ? cnt32[id] : c;
}

__device__ __forceinline__ void put_count(uint8_t *__restrict__ cnt8, uint32_t *__restrict__ cnt32,
                                          ull id, uint32_t c) {
  cnt8[id] = (uint8_t)(c < 255u ? c : 255u);
  if (c >= 255u) cnt32[id] = c;
}

// Arcs of the states of chunk c before state `id` (a state of that chunk,
// or the first state after it): summed by the whole workgroup, valid in
// thread 0.
__device__ __forceinline__ uint32_t chunk_arcs_before(const Problem &P, ull chunk, ull id,
                                                      const uint8_t *__restrict__ cnt8,
                                                      const uint32_t *__restrict__ cnt32,
                                                      uint32_t *s_w) {
  const ull first = P.wbase[chunk * OUT_WORDS];
  uint32_t part = 0;
  for (ull j = first + threadIdx.x; j < id; j += NT) part += count_of(cnt8, cnt32, j);
  return block_sum(part, s_w);
}

__device__ __forceinline__ uint32_t new_id(const Problem &P, uint32_t k) {
  const uint32_t w = k >> 5;
  return P.wbase[w] + (uint32_t)__popc(P.trim[w] & ((1u << (k & 31u)) - 1u));
}

__device__ __forceinline__ uint32_t out_units(const Fwd &s) { return s.eA + (uint32_t)s.be + s.mU; }

// A state of C (a trim key) that does not accept and has exactly one move:
// one epsilon move and no matching unit, or one non-epsilon arc on the
// smaller side whose label bucket on the other side holds at most one arc
// (that side's labels are distinct).  Its one move is a kept arc: a trim key
// that does not accept reaches an accepting key through some move, whose
// target is then co-accessible and, reached from an accessible key,
// accessible.  So its count is 1, known from its records alone.
__device__ __forceinline__ bool lone_move(const Fwd &s) {
  if (s.accept) return false;
  const uint32_t neps = s.eA + (uint32_t)s.be;
  if (neps == 1 && s.mU == 0) return true;
  if (neps != 0 || s.mU != 1) return false;
  return ((s.nA <= s.nB ? s.flB : s.flA) & (int32_t)FLAG_DISTINCT) != 0;
}

// The move of a state that has a single candidate: one epsilon arc and no
// matching unit, or no epsilon arc and one non-epsilon arc on the smaller
// side whose label bucket on the other side holds at most one arc.  Lanes of
// both kinds run the same straight-line loads, so a wavefront mixing them
// pays for one chain of dependent loads, not two.  `fast` is false when the
// state needs the general enumeration.
struct Move {
  bool fast, has;
  uint32_t d;
  int32_t il, ol;
  float w;
  int32_t pa, pb;
};

__device__ __forceinline__ Move single_move(const Problem &P, const Fwd &s) {
  Move m;
  m.fast = false;
  m.has = false;
  const uint32_t neps = s.eA + (uint32_t)s.be;
  const bool eps1 = neps == 1 && s.mU == 0;
  const bool m1 = neps == 0 && s.mU == 1;
  if (!eps1 && !m1) return m;
  int32_t pa = -1, pb = -1;
  uint32_t da, db, f = 0;
  if (eps1) {
    if (s.eA) {
      pa = s.aS;
      da = nbr_of(s.e0A);
      db = s.qb;
    } else {
      pb = s.bS;
      da = s.qa;
      db = nbr_of(s.e0B);
      f = s.epsA;
    }
  } else {
    int32_t lo, hi, nb0;
    if (s.nA <= s.nB) {
      pa = s.aS + s.ae;
      da = nbr_of(s.n1A);
      label_range(P.bOut, s.qb, s.bS + s.be, s.bE, s.l1A, lo, hi, nb0);
      pb = lo;
      db = nbr_of(nb0);
    } else {
      pb = s.bS + s.be;
      db = nbr_of(s.n1B);
      label_range(P.aOut, s.qa, s.aS + s.ae, s.aE, s.l1B, lo, hi, nb0);
      pa = lo;
      da = nbr_of(nb0);
    }
    if (hi - lo > 1) return m;  // several pairs: general enumeration
    m.fast = true;
    if (hi == lo) return m;  // no move
  }
  m.fast = true;
  m.has = true;
  m.d = make_key(da, db, f, P.shiftB);
  m.pa = pa;
  m.pb = pb;
  return m;
}

// The labels and weight of a single move.
__device__ __forceinline__ void move_labels(const Problem &P, Move &m) {
  const int32_t ia = m.pa >= 0 ? P.aOut.olab[m.pa] : 0;
  const float wa = m.pa >= 0 ? P.aOut.w[m.pa] : 0.f;
  const int32_t ob = m.pb >= 0 ? P.bOut.olab[m.pb] : 0;
  const float wb = m.pb >= 0 ? P.bOut.w[m.pb] : 0.f;
  m.il = ia;
  m.ol = ob;
  // epsilon arcs copy their weight (no + 0.0f, which would turn -0.0 into +0.0)
  m.w = (m.pa >= 0 && m.pb >= 0) ? wa + wb : (m.pa >= 0 ? wa : wb);
}

// Sequential enumeration of a state's moves in canonical order: A-epsilon
// arcs, B-epsilon arcs, then matching arcs by (label, a, b).  The join walks
// the label groups of the side with fewer non-epsilon arcs and looks up the
// other side's bucket; each group is emitted row-major (a outer, b inner).
// vis(target key, ilabel, olabel, weight, position in A's out-view or -1,
// position in B's out-view or -1).
template <class Visit>
__device__ __forceinline__ void enum_general(const Problem &P, const Fwd &s, Visit &&vis) {
  const uint32_t sh = P.shiftB;
  for (int32_t p = s.aS; p < s.aS + (int32_t)s.eA; ++p)
    vis(make_key(nbr_of(P.aOut.arec[p].y), s.qb, 0u, sh), P.aOut.olab[p], 0, P.aOut.w[p], p, -1);
  for (int32_t p = s.bS; p < s.bS + s.be; ++p)
    vis(make_key(s.qa, nbr_of(P.bOut.arec[p].y), s.epsA, sh), 0, P.bOut.olab[p], P.bOut.w[p], -1,
        p);
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
        const uint32_t da = nbr_of(P.aOut.arec[pa].y);
        const int32_t ia = P.aOut.olab[pa];
        const float wa = P.aOut.w[pa];
        for (int32_t pb = lo; pb < hi; ++pb)
          vis(make_key(da, nbr_of(P.bOut.arec[pb].y), 0u, sh), ia, P.bOut.olab[pb],
              wa + P.bOut.w[pb], pa, pb);
      }
      p = pend;
    }
  } else {
    // the first non-epsilon arc of qb comes from its record (no arc load)
    const int32_t p1 = s.bS + s.be;
    int32_t p = p1, al = s.aS + s.ae;
    while (p < s.bE) {
      const int32_t lab = p == p1 ? opaque(s.l1B) : P.bOut.arec[p].x;
      int32_t pend = p + 1;
      while (pend < s.bE && P.bOut.arec[pend].x == lab) ++pend;
      int32_t lo, hi, nb0;
      label_range(P.aOut, s.qa, al, s.aE, lab, lo, hi, nb0);
      if (lo < hi) al = hi;
      for (int32_t pa = lo; pa < hi; ++pa) {
        const uint32_t da = nbr_of(pa == lo ? nb0 : P.aOut.arec[pa].y);
        const int32_t ia = P.aOut.olab[pa];
        const float wa = P.aOut.w[pa];
        for (int32_t pb = p; pb < pend; ++pb)
          vis(make_key(da, nbr_of(pb == p1 ? opaque(s.n1B) : P.bOut.arec[pb].y), 0u, sh), ia,
              P.bOut.olab[pb], wa + P.bOut.w[pb], pa, pb);
      }
      p = pend;
    }
  }
}

template <class Visit>
__device__ __forceinline__ void enum_light(const Problem &P, const Fwd &s, Visit &&vis) {
  Move m = single_move(P, s);
  if (m.fast) {
    if (m.has) {
      move_labels(P, m);
      vis(m.d, m.il, m.ol, m.w, m.pa, m.pb);
    }
    return;
  }
  enum_general(P, s, vis);
}

// Output of C is written once and not read back here: streaming stores
// (no allocation in the caches; 7 % faster fill).
template <class T>
__device__ __forceinline__ void out_store(T *p, T v) {
  __builtin_nontemporal_store(v, p);
}

// Write one arc of C if its target dk is a trim key; pa / pb are positions
// in the out-views (-1: none), turned into arc ids only when provenance is
// requested.  Every load (the target's trim word and prefix, the arc ids)
// is issued before the test and the stores, so they share one round trip.
__device__ __forceinline__ bool put_arc(const OutGraph &O, const Problem &P, uint32_t pos,
                                        uint32_t id, uint32_t dk, int32_t il, int32_t ol,
                                        float w, int32_t pa, int32_t pb) {
  const uint32_t tw = P.trim[dk >> 5], base = P.wbase[dk >> 5];
  const int32_t ida = O.arc_a && pa >= 0 ? P.aOut.perm[pa] + O.aebase : -1;
  const int32_t idb = O.arc_b && pb >= 0 ? P.bOut.perm[pb] : -1;
  const uint32_t below = tw & ((1u << (dk & 31u)) - 1u);
  if (!((tw >> (dk & 31u)) & 1u)) return false;
  out_store(O.src + pos, (int32_t)id + O.vbase);
  out_store(O.dst + pos, (int32_t)(base + (uint32_t)__popc(below)) + O.vbase);
  out_store(O.il + pos, il);
  out_store(O.ol + pos, ol);
  out_store(O.w + pos, w);
  if (O.arc_a) out_store(O.arc_a + pos, ida);
  if (O.arc_b) out_store(O.arc_b + pos, idb);
  return true;
}

// put_arc for a single move: the target's trim word and prefix, the arc ids
// and the move's labels and weights are all loaded in one round trip.
__device__ __forceinline__ void put_move(const OutGraph &O, const Problem &P, uint32_t pos,
                                         uint32_t id, Move m) {
  const uint32_t dk = m.d;
  const uint32_t tw = P.trim[dk >> 5], base = P.wbase[dk >> 5];
  const int32_t ida = O.arc_a && m.pa >= 0 ? P.aOut.perm[m.pa] + O.aebase : -1;
  const int32_t idb = O.arc_b && m.pb >= 0 ? P.bOut.perm[m.pb] : -1;
  move_labels(P, m);
  const uint32_t below = tw & ((1u << (dk & 31u)) - 1u);
  if (!((tw >> (dk & 31u)) & 1u)) return;
  out_store(O.src + pos, (int32_t)id + O.vbase);
  out_store(O.dst + pos, (int32_t)(base + (uint32_t)__popc(below)) + O.vbase);
  out_store(O.il + pos, m.il);
  out_store(O.ol + pos, m.ol);
  out_store(O.w + pos, m.w);
  if (O.arc_a) out_store(O.arc_a + pos, ida);
  if (O.arc_b) out_store(O.arc_b + pos, idb);
}

// Workgroup-cooperative canonical enumeration of one heavy state.  Every
// thread of the workgroup must call it.  Returns the number of kept arcs;
// with FILL it also writes them from arc position `pos0` on.
template <bool FILL>
__device__ uint32_t heavy_state(const Problem &P, uint32_t id, uint32_t key, uint32_t pos0,
                                const OutGraph &O, uint32_t *s_w) {
  const Fwd s = fwd_info<false>(P, key);
  const uint32_t sh = P.shiftB;
  const unsigned t = threadIdx.x;
  uint32_t run = 0;
  for (uint32_t c = 0; c < s.eA; c += NT) {
    const uint32_t i = c + t;
    bool keep = false;
    int32_t pa = 0;
    uint32_t d = 0;
    if (i < s.eA) {
      pa = s.aS + (int32_t)i;
      d = make_key(nbr_of(P.aOut.arec[pa].y), s.qb, 0u, sh);
      keep = test_bit(P.trim, d);
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan<uint32_t>(keep ? 1u : 0u, s_w, tot);
    if (FILL && keep)
      put_arc(O, P, pos0 + run + ex, id, d, P.aOut.olab[pa], 0, P.aOut.w[pa], pa, -1);
    run += tot;
  }
  for (uint32_t c = 0; c < (uint32_t)s.be; c += NT) {
    const uint32_t i = c + t;
    bool keep = false;
    int32_t pb = 0;
    uint32_t d = 0;
    if (i < (uint32_t)s.be) {
      pb = s.bS + (int32_t)i;
      d = make_key(s.qa, nbr_of(P.bOut.arec[pb].y), s.epsA, sh);
      keep = test_bit(P.trim, d);
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan<uint32_t>(keep ? 1u : 0u, s_w, tot);
    if (FILL && keep)
      put_arc(O, P, pos0 + run + ex, id, d, 0, P.bOut.olab[pb], P.bOut.w[pb], -1, pb);
    run += tot;
  }
  if (s.mU) {
    // A-driven: A's non-epsilon arcs in (label, a) order, each joined with
    // B's bucket of its label, gives (label, a, b) order.
    for (uint32_t c = 0; c < s.nA; c += NT) {
      const uint32_t i = c + t;
      int32_t lo = 0, hi = 0, pa = 0;
      uint32_t kept = 0, da = 0;
      if (i < s.nA) {
        pa = s.aS + s.ae + (int32_t)i;
        const int2 ar = P.aOut.arec[pa];
        da = nbr_of(ar.y);
        label_range(P.bOut, s.qb, s.bS + s.be, s.bE, ar.x, lo, hi);
        for (int32_t pb = lo; pb < hi; ++pb)
          kept += test_bit(P.trim, make_key(da, nbr_of(P.bOut.arec[pb].y), 0u, sh));
      }
      uint32_t tot;
      uint32_t ex = block_excl_scan<uint32_t>(kept, s_w, tot);
      if (FILL && kept) {
        const int32_t ia = P.aOut.olab[pa];
        const float wa = P.aOut.w[pa];
        uint32_t pos = pos0 + run + ex;
        for (int32_t pb = lo; pb < hi; ++pb) {
          const uint32_t d = make_key(da, nbr_of(P.bOut.arec[pb].y), 0u, sh);
          if (test_bit(P.trim, d))
            put_arc(O, P, pos++, id, d, ia, P.bOut.olab[pb], wa + P.bOut.w[pb], pa, pb);
        }
      }
      run += tot;
    }
  }
  return run;
}

// The kept-arc count of a heavy state (the same moves as heavy_state): each
// thread counts its share of the moves, one block sum at the end; valid in
// thread 0.  Every thread of the workgroup must call it.
__device__ uint32_t heavy_count(const Problem &P, uint32_t key, uint32_t *s_w) {
  const Fwd s = fwd_info<false>(P, key);
  const uint32_t sh = P.shiftB;
  uint32_t kept = 0;
#pragma unroll 4
  for (uint32_t i = threadIdx.x; i < s.eA; i += NT)
    kept += test_bit(P.trim, make_key(nbr_of(P.aOut.arec[s.aS + (int32_t)i].y), s.qb, 0u, sh));
#pragma unroll 4
  for (uint32_t i = threadIdx.x; i < (uint32_t)s.be; i += NT)
    kept += test_bit(P.trim, make_key(s.qa, nbr_of(P.bOut.arec[s.bS + (int32_t)i].y), s.epsA, sh));
  if (s.mU)
    for (uint32_t i = threadIdx.x; i < s.nA; i += NT) {
      const int2 ar = P.aOut.arec[s.aS + s.ae + (int32_t)i];
      const uint32_t da = nbr_of(ar.y);
      int32_t lo, hi;
      label_range(P.bOut, s.qb, s.bS + s.be, s.bE, ar.x, lo, hi);
      for (int32_t pb = lo; pb < hi; ++pb)
        kept += test_bit(P.trim, make_key(da, nbr_of(P.bOut.arec[pb].y), 0u, sh));
    }
  return block_sum(kept, s_w);
}

// Kept-arc counts, one output chunk per wavefront: put_count for light
// states (0 for now for heavy ones, which are listed with their keys), and
// btot[chunk] = the chunk's light total.
__global__ __launch_bounds__(NT) void k_count(Problem P, ull nwords, ull nchunks,
                                              uint8_t *__restrict__ cnt8,
                                              uint32_t *__restrict__ cnt32,
                                              uint32_t *__restrict__ btot,
                                              uint2 *__restrict__ heavy, Scalars *sc) {
  const ull chunk = (ull)blockIdx.x * NWAVES + threadIdx.x / WAVE;
  if (chunk >= nchunks) return;  // the whole wavefront
  __shared__ uint16_t s_keys[NWAVES][OUT_WORDS * 32];
  uint16_t *list = s_keys[threadIdx.x / WAVE];
  const TrimChunk t = trim_chunk(P, chunk, nwords);
  const uint32_t first = t.count ? P.wbase[t.w0] : 0u;
  trim_expand(t, list);
  uint32_t sum = 0;
  // each round reads the next round's keys before its own loads
  uint32_t key_next = trim_key_at(t, list, __lane_id());
  for (uint32_t i0 = 0; i0 < t.count; i0 += WAVE) {
    const uint32_t i = i0 + __lane_id();
    const uint32_t key = key_next;
    key_next = trim_key_at(t, list, i + WAVE);
    bool hv = false;
    if (i < t.count) {
      const Fwd s = fwd_info(P, key);
      uint32_t c = 0;
      if (out_units(s) > LIGHT_UNITS) {
        hv = true;
      } else if (lone_move(s)) {
        c = 1;
      } else {
        enum_light(P, s, [&](uint32_t d, int32_t, int32_t, float, int32_t, int32_t) {
          c += test_bit(P.trim, d) ? 1u : 0u;
        });
      }
      put_count(cnt8, cnt32, (ull)first + i, c);
      sum += c;
    }
    unsigned long long m = __ballot(hv);
    if (m) {
      const int leader = __ffsll(m) - 1;
      uint32_t hb = 0;
      if ((int)__lane_id() == leader) hb = atomicAdd(&sc->heavy, (uint32_t)__popcll(m));
      hb = __shfl(hb, leader, WAVE);
      if (hv) heavy[hb + __popcll(m & __lanemask_lt())] = make_uint2(first + i, key);
    }
  }
  sum = wave_sum(sum);
  if (__lane_id() == 0) btot[chunk] = sum;
}

// Counts of the heavy states (one workgroup each), added to their chunk's
// btot.
__global__ __launch_bounds__(NT) void k_count_heavy(Problem P, const uint2 *__restrict__ heavy,
                                                    const uint32_t *__restrict__ nheavy_p,
                                                    uint8_t *__restrict__ cnt8,
                                                    uint32_t *__restrict__ cnt32,
                                                    uint32_t *__restrict__ btot) {
  __shared__ uint32_t s_w[NWAVES];
  const uint32_t nheavy = *nheavy_p;
  for (uint32_t h = blockIdx.x; h < nheavy; h += gridDim.x) {
    const uint2 hk = heavy[h];
    const uint32_t c = heavy_count(P, hk.y, s_w);
    if (threadIdx.x == 0) {
      put_count(cnt8, cnt32, hk.x, c);
      atomicAdd(btot + (hk.y >> 5) / OUT_WORDS, c);
    }
    __syncthreads();  // s_w is read by thread 0 before the next state's sum
  }
}

// One thread per state of C, one output chunk per wavefront: the state's
// arc offset (chunk offset + wavefront scan of the counts), flags and key,
// and the arcs of a light state (heavy states are written by the
// workgroups of k_fill set aside for them).
__device__ __forceinline__ void fill_light(const Problem &P, ull nwords, ull nchunks,
                                           const uint8_t *__restrict__ cnt8,
                                           const uint32_t *__restrict__ cnt32,
                                           const uint32_t *__restrict__ btot,
                                           const OutGraph &O, unsigned block) {
  const ull chunk = (ull)block * NWAVES + threadIdx.x / WAVE;
  if (chunk >= nchunks) return;  // the whole wavefront
  __shared__ uint16_t s_keys[NWAVES][OUT_WORDS * 32];
  uint16_t *list = s_keys[threadIdx.x / WAVE];
  const TrimChunk t = trim_chunk(P, chunk, nwords);
  if (!t.count) return;
  const uint32_t first = P.wbase[t.w0], end = first + t.count;
  uint32_t run = btot[chunk];
  trim_expand(t, list);
  // rounds cover ids [64 k, 64 k + 64), so that the state outputs of a
  // round (offsets, flags) fill whole aligned segments; lanes outside the
  // chunk are idle
  const uint32_t a0 = first & ~(uint32_t)(WAVE - 1);
  uint32_t c_next = 0, key_next = 0;
  {
    const uint32_t id = a0 + __lane_id();
    if (id >= first && id < end) {
      c_next = count_of(cnt8, cnt32, id);
      key_next = trim_key_at(t, list, id - first);
    }
  }
  for (uint32_t g0 = a0; g0 < end; g0 += WAVE) {
    const uint32_t id = g0 + __lane_id();
    const bool valid = id >= first && id < end;
    const uint32_t c = c_next, key = key_next;
    const uint32_t nid = id + WAVE;
    if (nid >= first && nid < end) {
      c_next = count_of(cnt8, cnt32, nid);
      key_next = trim_key_at(t, list, nid - first);
    }
    const uint32_t incl = wave_incl_scan(c);
    uint32_t pos = run + incl - c;
    run += __shfl(incl, WAVE - 1, WAVE);
    if (!valid) continue;
    const Fwd s = fwd_info(P, key);
    out_store(O.arc_offset + id, (int32_t)pos + O.ebase);
    out_store(O.accept + id, (uint8_t)(s.accept ? 1 : 0));
    out_store(O.start + id, (uint8_t)(s.start ? 1 : 0));
    if (O.key_a) out_store(O.key_a + id, (int32_t)s.qa + O.abase);
    if (O.key_b) out_store(O.key_b + id, (int32_t)s.qb);
    if (O.key_f) out_store(O.key_f + id, (uint8_t)s.f);
    if (out_units(s) > LIGHT_UNITS) continue;
    const Move m = single_move(P, s);
    if (m.fast) {
      if (m.has) put_move(O, P, pos, id, m);
    } else {
      enum_general(P, s, [&](uint32_t d, int32_t il, int32_t ol, float w, int32_t pa, int32_t pb) {
        if (put_arc(O, P, pos, id, d, il, ol, w, pa, pb)) ++pos;
      });
    }
  }
}

// The fill in one launch: workgroups [0, hb) write the heavy states (one
// workgroup per state, the heavy list strided over them), the others the
// light chunks, so the heavy states' workgroup loops run under the light
// work.  A heavy state's first arc position is its chunk's offset plus the
// counts of the chunk's earlier states, summed by its workgroup.
__global__ __launch_bounds__(NT) void k_fill(Problem P, ull nwords, ull nchunks,
                                             const uint8_t *__restrict__ cnt8,
                                             const uint32_t *__restrict__ cnt32,
                                             const uint32_t *__restrict__ btot, uint32_t nstates,
                                             uint32_t narcs, const uint2 *__restrict__ heavy,
                                             uint32_t nheavy, unsigned hb, OutGraph O) {
  if (blockIdx.x < hb) {
    __shared__ uint32_t s_w[NWAVES];
    __shared__ uint32_t s_pos;
    for (uint32_t h = blockIdx.x; h < nheavy; h += hb) {
      const uint2 hk = heavy[h];
      const ull chunk = (hk.y >> 5) / OUT_WORDS;
      const uint32_t before = chunk_arcs_before(P, chunk, hk.x, cnt8, cnt32, s_w);
      if (threadIdx.x == 0) s_pos = btot[chunk] + before;
      __syncthreads();
      heavy_state<true>(P, hk.x, hk.y, s_pos, O, s_w);
      __syncthreads();  // s_pos and s_w are reused by the next heavy state
    }
    return;
  }
  const unsigned block = blockIdx.x - hb;
  fill_light(P, nwords, nchunks, cnt8, cnt32, btot, O, block);
  if (block == gridDim.x - hb - 1 && threadIdx.x == 0)
    O.arc_offset[nstates] = (int32_t)narcs + O.ebase;
}

// ---------------------------------------------------------------------------
// batches: the disjoint union of several A, and each item's range in C
// ---------------------------------------------------------------------------

// Item graph a at state offset vbase and arc offset ebase of the union:
// offsets, sources and destinations shifted (labels, weights and flags are
// copied as they are).
__global__ __launch_bounds__(NT) void k_union_copy(DevGraph a, long long vbase, long long ebase,
                                                   int32_t *__restrict__ off,
                                                   int32_t *__restrict__ src,
                                                   int32_t *__restrict__ dst) {
  const long long n = (long long)a.V + 1 > (long long)a.E ? (long long)a.V + 1 : (long long)a.E;
  for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < n;
       i += (long long)gridDim.x * NT) {
    if (i <= a.V) off[vbase + i] = (int32_t)(a.off[i] + ebase);
    if (i < a.E) {
      src[ebase + i] = (int32_t)(a.src[i] + vbase);
      dst[ebase + i] = (int32_t)(a.dst[i] + vbase);
    }
  }
}

// out[i] = first state of item i in C (the number of trim keys below the
// item's first key), out[n + 1 + i] = its first arc (the chunk's arc offset
// plus the counts of the chunk's earlier states, summed by the workgroup of
// the item), for i <= n.
__global__ __launch_bounds__(NT) void k_item_ranges(Problem P, ull nkeys, int32_t n,
                                                    const long long *__restrict__ qa_base,
                                                    const uint8_t *__restrict__ cnt8,
                                                    const uint32_t *__restrict__ cnt32,
                                                    const uint32_t *__restrict__ btot,
                                                    uint32_t nstates, uint32_t narcs,
                                                    long long *__restrict__ out) {
  __shared__ uint32_t s_w[NWAVES];
  for (int i = blockIdx.x; i <= n; i += gridDim.x) {
    const ull K = (ull)qa_base[i] << (P.shiftB + 1);
    const uint32_t st = K >= nkeys ? nstates : new_id(P, (uint32_t)K);
    // the item's first state is the first trim key >= K: a state of K's
    // chunk, or the first state after it
    const ull chunk = (K >> 5) / OUT_WORDS;
    uint32_t before = 0;
    if (st < nstates) before = chunk_arcs_before(P, chunk, st, cnt8, cnt32, s_w);
    if (threadIdx.x == 0) {
      out[i] = st;
      out[n + 1 + i] = st < nstates ? (long long)(btot[chunk] + before) : (long long)narcs;
    }
    __syncthreads();  // s_w is reused by the next item
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_validate(const DevGraph &g, int side, uint32_t *err, uint32_t *maxlab,
                           hipStream_t s, uint32_t *nacc, bool check) {
  size_t n = (size_t)(g.V + 1 > g.E ? g.V + 1 : g.E);
  if (check) k_validate<<<grid_for(n, 2048), NT, 0, s>>>(g, side, err, maxlab, nacc);
  else k_label_facts<<<grid_for(n, 2048), NT, 0, s>>>(g, side, err, maxlab, nacc);
  return hipGetLastError();
}

hipError_t sort_view(const DevGraph &g, int side, bool by_dst, bool presorted, int lab_bits,
                     int4 *srec, int2 *arec, int32_t *perm, int32_t *olab, float *w,
                     int32_t *off_tmp, const int4 *eps_rec, unsigned long long *k0, int32_t *v0,
                     unsigned long long *k1, int32_t *v1, void *sort_temp, uint32_t *eps_states,
                     hipStream_t s) {
  const size_t E = (size_t)g.E;
  hipError_t e;
  if (E) {
    const bool sort = by_dst || !presorted;
    bool second = false;
    if (sort) {
      k_make_keys<<<grid_for(E), NT, 0, s>>>(g, side, by_dst ? 1 : 0, lab_bits, k0, v0);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      int bits = bitlen((unsigned long long)(g.V > 0 ? g.V - 1 : 0)) + lab_bits;
      if ((e = radix_sort(k0, v0, k1, v1, E, bits, sort_temp, s, &second)) != hipSuccess)
        return e;
    }
    const ull *ks = sort ? (second ? k1 : k0) : nullptr;
    const int32_t *vs = sort ? (second ? v1 : v0) : nullptr;
    k_split<<<grid_for(E), NT, 0, s>>>(g, by_dst ? 1 : 0, ks, vs, (long long)E, lab_bits, eps_rec,
                                       side, perm, olab, w, arec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (by_dst) {
      if (4 * E >= (size_t)g.V)
        k_group_bounds<<<grid_for(E + 1, 2048), NT, 0, s>>>(ks, (long long)E, g.V, lab_bits,
                                                           off_tmp);
      else
        k_group_offsets<<<grid_for((size_t)g.V + 1), NT, 0, s>>>(ks, (long long)E, g.V,
                                                                lab_bits, off_tmp);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  } else if (by_dst) {
    k_group_offsets<<<grid_for((size_t)g.V + 1), NT, 0, s>>>(nullptr, 0, g.V, lab_bits, off_tmp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int32_t *off = by_dst ? off_tmp : g.off;
  if (g.V) {
    const int eps_mode = side == 1 ? 0 : (by_dst ? 2 : 1);
    k_state_rec<<<grid_for((size_t)g.V, 256), NT, 0, s>>>(off, arec, g.V, g.accept,
                                                          by_dst ? nullptr : g.start, eps_mode,
                                                          eps_rec, srec, eps_states);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t finish_views(ViewJobs J, hipStream_t s) {
  hipError_t e;
  if (J.vbegin[4]) {
    k_mark_unique<<<grid_for((size_t)J.vbegin[4]), NT, 0, s>>>(J);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (J.ebegin[4]) {
    k_mark_arcs<<<grid_for((size_t)J.ebegin[4]), NT, 0, s>>>(J);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (J.vbegin[4]) {
    k_state_inline<<<grid_for((size_t)J.vbegin[4]), NT, 0, s>>>(J);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (J.j[0].chain || J.j[1].chain || J.j[2].chain || J.j[3].chain) {
      k_chains<<<grid_for((size_t)J.vbegin[4]), NT, 0, s>>>(J);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  if (J.lbegin[4]) {
    k_build_lut<<<grid_for((size_t)J.lbegin[4], 8192), NT, 0, s>>>(J);
    if ((e = hipGetLastError()) != hipSuccess) return e;
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

hipError_t launch_seed_backward_all(const Problem &P, const SearchArgs &S, int32_t *la,
                                    uint32_t *na, int32_t *lb, uint32_t *nb, hipStream_t s) {
  k_collect<<<grid_for((size_t)P.A.V, 1024), NT, 0, s>>>(P.A.accept, P.A.V, la, na);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_collect<<<grid_for((size_t)P.B.V, 1024), NT, 0, s>>>(P.B.accept, P.B.V, lb, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_seed_backward_all<<<1024, NT, 0, s>>>(P, S, la, na, lb, nb);
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

hipError_t launch_generation2(const Problem &P, const SearchArgs &SF, const SearchArgs &SB, int gf,
                              int gb, hipStream_t s) {
  constexpr unsigned GRID = 1024;
  k_gen2<<<2 * GRID, NT, 0, s>>>(P, SF, SB, gf, gb);
  return hipGetLastError();
}

hipError_t launch_count_moves(const Problem &P, size_t nwords, bool forward,
                              unsigned long long *out, hipStream_t s) {
  if (!nwords) return hipSuccess;
  const unsigned g = grid_for(nwords * 32, 1u << 17);
  if (forward) k_count_moves<true><<<g, NT, 0, s>>>(P, nwords, out);
  else k_count_moves<false><<<g, NT, 0, s>>>(P, nwords, out);
  return hipGetLastError();
}

hipError_t launch_popcount(const uint32_t *bm, size_t nwords, unsigned long long *out,
                           hipStream_t s) {
  if (!nwords) return hipSuccess;
  // few workgroups: each adds its sum with one atomic on the same counter
  k_popcount<<<grid_for(nwords / 4 + 1, 256), NT, 0, s>>>(bm, nwords, out);
  return hipGetLastError();
}

hipError_t launch_trim(const Problem &P, uint32_t VA, uint32_t *trim, uint32_t *cnt,
                       hipStream_t s) {
  if (!VA) return hipSuccess;
  const uint32_t ntA = (VA + TRIM_ROWS - 1) / TRIM_ROWS;
  const ull WR = ((ull)P.maskB + 1) >> 4, ntB = (WR + 15) / 16;
  const ull ntiles = (ull)ntA * ntB;
  // a multiple of 8 workgroups (one share per XCD), at most 8 x 2048
  const ull per = (ntiles + 7) / 8;
  const unsigned grid = (unsigned)(8 * (per < 2048 ? per : 2048));
  k_trim<<<grid, NT, 0, s>>>(P, VA, ntA, ntiles, trim, cnt);
  return hipGetLastError();
}

hipError_t launch_count(const Problem &P, size_t nwords, uint8_t *cnt8, uint32_t *cnt32,
                        uint32_t *btot, uint2 *heavy, Scalars *sc, hipStream_t s) {
  const size_t nchunks = out_chunks(nwords);
  if (!nchunks) return hipSuccess;
  if (!P.trim || !P.wbase) return hipErrorInvalidValue;  // no trim bitmap to expand
  k_count<<<out_grid(nchunks), NT, 0, s>>>(P, nwords, nchunks, cnt8, cnt32, btot, heavy, sc);
  return hipGetLastError();
}

hipError_t launch_count_heavy(const Problem &P, const uint2 *heavy, const uint32_t *nheavy_dev,
                              uint8_t *cnt8, uint32_t *cnt32, uint32_t *btot, hipStream_t s) {
  k_count_heavy<<<1024, NT, 0, s>>>(P, heavy, nheavy_dev, cnt8, cnt32, btot);
  return hipGetLastError();
}

hipError_t launch_fill(const Problem &P, size_t nwords, const uint8_t *cnt8,
                       const uint32_t *cnt32, const uint32_t *btot, const uint2 *heavy,
                       uint32_t nheavy, uint32_t nstates, uint32_t narcs, const OutGraph &O,
                       hipStream_t s) {
  const size_t nchunks = out_chunks(nwords);
  if (nchunks && (!P.trim || !P.wbase)) return hipErrorInvalidValue;  // no trim bitmap
  const unsigned hb = nheavy < 4096 ? nheavy : 4096;
  k_fill<<<hb + out_grid(nchunks), NT, 0, s>>>(P, nwords, nchunks, cnt8, cnt32, btot, nstates,
                                               narcs, heavy, nheavy, hb, O);
  return hipGetLastError();
}

hipError_t launch_union_copy(const DevGraph &a, long long vbase, long long ebase, int32_t *off,
                             int32_t *src, int32_t *dst, hipStream_t s) {
  const size_t n = (size_t)(a.V + 1 > a.E ? a.V + 1 : a.E);
  k_union_copy<<<grid_for(n), NT, 0, s>>>(a, vbase, ebase, off, src, dst);
  return hipGetLastError();
}

hipError_t launch_item_ranges(const Problem &P, unsigned long long nkeys, int32_t n,
                              const long long *qa_base, const uint8_t *cnt8,
                              const uint32_t *cnt32, const uint32_t *btot, uint32_t nstates,
                              uint32_t narcs, long long *out, hipStream_t s) {
  const unsigned g = (unsigned)(n + 1 < 4096 ? n + 1 : 4096);
  k_item_ranges<<<g, NT, 0, s>>>(P, nkeys, n, qa_base, cnt8, cnt32, btot, nstates, narcs, out);
  return hipGetLastError();
}

}  // namespace fstc
