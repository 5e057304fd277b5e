// Internal declarations shared by the HIP translation units of
// libfstcompose.so.  Device code targets gfx950 (CDNA4, 64-wide wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fst_compose.h"

namespace fstc {

constexpr int NT = 256;              // threads per workgroup (4 wavefronts)
constexpr int WAVE = 64;             // CDNA wavefront width
constexpr int NWAVES = NT / WAVE;
constexpr uint32_t LIGHT_UNITS = 32;   // compaction: per-state work above this goes to a workgroup
constexpr uint32_t LIGHT_SEARCH = 64;  // search: a key with more units is split over threads
constexpr int CHAIN_MAX = 64;          // search: default depth-first budget per thread
constexpr uint32_t NO_KEY = 0xFFFFFFFFu;

// The output passes give every wavefront one chunk of OUT_WORDS consecutive
// trim words (its states are consecutive ids), so the arcs a wavefront
// writes are contiguous and its offsets need only wavefront scans.  Every
// workgroup covers NWAVES consecutive chunks.
constexpr size_t OUT_WORDS = 16;
inline size_t out_chunks(size_t nwords) { return (nwords + OUT_WORDS - 1) / OUT_WORDS; }
inline unsigned out_grid(size_t nchunks) {
  const size_t g = (nchunks + NWAVES - 1) / NWAVES;
  return (unsigned)(g ? g : 1);
}

// ---------------------------------------------------------------------------
// Graph views
// ---------------------------------------------------------------------------

// The caller's structure-of-arrays graph (Section 3.2), device pointers.
struct DevGraph {
  int32_t V, E;
  const int32_t *off, *src, *dst, *il, *ol;
  const float *w;
  const uint8_t *start, *accept;
};

// Arcs grouped by a state (their source for out-views, their destination for
// in-views) and sorted inside each group by the matched label, ties by arc id.
// Label 0 (epsilon) sorts first, so a group starts with its epsilon arcs.
//   srec[2v]   = {group begin, epsilon arcs, group end, flags}: FLAG_ACCEPT
//                is accept(v); in views of A, FLAG_EPS_OUT is epsOutA(v) (v
//                has an out-arc with output epsilon); in out-views
//                FLAG_START is start(v); FLAG_UNIQ, see below.
//   srec[2v+1] = {other end of the group's first epsilon arc, label and
//                other end of its first non-epsilon arc, 0} (arec fields,
//                0 where there is no such arc): the 32-byte record of a
//                state with one arc of a kind resolves that arc without an
//                arc-record load.
//   arec[i] = {matched label, other end}: the destination in out-views, the
//             source in in-views (NBR_MASK bits); NBR_UNIQ is the other end's
//             FLAG_UNIQ in this view; in A's in-view NBR_EPS carries
//             epsOutA(source).
//   FLAG_UNIQ in an out-view marks a state that guarantees any key holding
//   it has at most one incoming move (in B: not a start state and exactly
//   one in-arc; in A: not a start state, no epsilon output, and in-arcs with
//   distinct non-epsilon output labels from states without epsilon output).
//   In an in-view it marks at most one outgoing move (in B: not accepting,
//   exactly one out-arc; in A: not accepting, no epsilon in-arc, out-arcs
//   with distinct non-epsilon output labels).  A key whose two states are
//   both marked is reached once by a search in that direction, so it needs
//   no claim.
//   FLAG_DISTINCT marks a state whose non-epsilon arcs in the view all have
//   different labels (checked for groups of at most DISTINCT_SCAN_MAX
//   non-epsilon arcs; larger groups are left unmarked), so any label bucket
//   of the state holds at most one arc.
//   chain (views of B, optional): per state, up to CHAIN_STEPS steps of its
//   single-arc path in the view: {n, l0, s0, l1, s1, ..., l10, s10} as
//   CHAIN_INT4 int4, where step i follows the only arc (label l_i, non-epsilon) of the
//   state reached after i steps to s_i (an arc-record neighbour field with
//   NBR_UNIQ), and a step is recorded only while the state it leaves has
//   exactly one arc in the view (in out-views: and is not accepting).
//   perm[i] = original arc id.
//   olab[i], w[i] (out-views only) = the arc's label on the output side of
//             the composition (A: input label, B: output label) and its
//             weight, gathered into sorted order for writing C.
//   lut, when present, holds every group's label buckets:
//             lut[v * lstride + l] = {begin, end, other end of the first arc,
//             0} for label l in group v, so a one-arc bucket resolves its
//             neighbour in a single lookup.
struct View {
  const int4 *srec;
  const int2 *arec;
  const int32_t *perm;
  const int4 *lut;
  int32_t lstride;  // largest label + 1
  const int32_t *olab;
  const float *w;
  const int4 *chain;
};

constexpr int CHAIN_STEPS = 11;
constexpr int CHAIN_INT4 = (1 + 2 * CHAIN_STEPS + 3) / 4;  // int4 per chain record

constexpr uint32_t FLAG_ACCEPT = 1u, FLAG_EPS_OUT = 2u, FLAG_START = 4u, FLAG_UNIQ = 8u,
                   FLAG_DISTINCT = 16u;
constexpr int32_t DISTINCT_SCAN_MAX = 256;
constexpr int32_t NBR_MASK = 0x3fffffff;            // state ids < 2^30
constexpr int32_t NBR_UNIQ = 0x40000000;
constexpr int32_t NBR_EPS = (int32_t)0x80000000u;

// Everything a search / compaction kernel needs, passed by value.
struct Problem {
  DevGraph A, B;
  View aOut;   // A by (src, olabel)
  View bOut;   // B by (src, ilabel)
  View aIn;    // A by (dst, olabel)
  View bIn;    // B by (dst, ilabel)
  uint32_t shiftB;        // bits of the B state inside a key
  int chain_max;          // keys one search thread may follow depth-first
  int restrict_fwd;       // forward search expands only keys already in coacc
  int restrict_bwd;       // backward search expands only keys already in vis
  int mark_accept;        // forward search marks accepting keys co-accessible
                          // and lists them as backward seeds
  // The two search bitmaps use the diagonal layout of search_bit(): a key
  // (qa, qb, f) sits at bit 2 (d rowA + qa) + f with d = (qb - qa) mod
  // 2^shiftB, so the keys of a chain that advances both states by one share
  // a bitmap word.  The trim bitmap is in key order (bit = key).
  uint32_t maskB;         // 2^shiftB - 1
  uint32_t rowA;          // A states per diagonal, rounded up to 16
  uint32_t *vis;          // accessible keys (search layout)
  uint32_t *coacc;        // co-accessible keys (search layout)
  const uint32_t *trim;   // accessible and co-accessible keys (key order)
  const uint32_t *wbase;  // exclusive popcount prefix of trim words
};

// Output arrays of C.  The arrays may start inside a larger C (one part of
// a batch): written ids then add vbase (states), ebase (arc offsets), abase
// (key_a, A states) and aebase (arc_a, A arcs); all 0 otherwise.
struct OutGraph {
  int32_t *arc_offset, *src, *dst, *il, *ol;
  float *w;
  uint8_t *start, *accept;
  int32_t *key_a, *key_b;
  uint8_t *key_f;
  int32_t *arc_a, *arc_b;
  int32_t vbase, ebase, abase, aebase;
};

// Work of one search generation, kept in one of three rotating slots
// (generation g uses slot g % 3): frontier keys Q[qbase, qbase + qcount) and
// heavy keys heavy[hbase, hbase + count) with their unit offsets, where
// hpack = (total units << 32) | count.  Generation g fills the slot of g + 1
// and clears the slot of g + 2.
struct GenSlot {
  uint32_t qbase, qcount, hbase, pad;
  unsigned long long hpack;
};

// Device scalars read back by the host (one pinned mirror).
struct Scalars {
  uint32_t errA, errB;          // validation error bits
  uint32_t maxLabA, maxLabB;    // max matched label (A olabel, B ilabel)
  uint32_t nEpsStatesA;         // states of A with an epsilon-output arc
  uint32_t tail2;               // accepting keys found by the forward search
  uint32_t naccA, naccB;        // accepting states of A and B
  uint32_t pad0;
  uint32_t heavy;               // heavy states of C
  uint32_t overflow;            // a capacity was exceeded
  uint32_t gens;                // search generations that had work
  uint32_t pad2;
  unsigned long long generated; // moves out of accessible keys (on request)
  unsigned long long generated_bwd; // predecessor moves of co-accessible keys (on request)
  unsigned long long naccessible; // keys reached by the forward search
  unsigned long long total;     // scan totals
  GenSlot G[3];                 // generation slots of a search
  GenSlot G2[3];                // of the backward search running beside it
  uint32_t gens2, pad1;         // its generations that had work
};

// Arrays of one search (each holds up to `cap` keys).
struct SearchArgs {
  uint32_t *Q;      // frontier keys, generation after generation
  uint32_t *heavy;  // heavy keys, generation after generation
  uint32_t *hoff;   // unit offset of each heavy key inside its generation
  uint32_t *acc;    // forward search: accepting keys, the backward seeds
  uint32_t cap;
  Scalars *sc;
  GenSlot *G;       // this search's three generation slots
  uint32_t *gens;   // this search's count of generations that had work
};

// ---------------------------------------------------------------------------
// Three inputs, C = A o B o D (compose3.hip)
// ---------------------------------------------------------------------------

// Everything the three-input kernels read, passed by value.  Keys are
// ((((qa << shB | qb) << 1 | f1) << shD | qd) << 1 | f2), 64-bit; a key's
// state is named by its slot in the hash set tab (hmask + 1 slots, empty =
// all ones) until the numbering.
struct Problem3 {
  DevGraph A, B, D;
  View aOut;  // A by (src, olabel), with A's ilabel and weight in sorted order
  View bOut;  // B by (src, ilabel), with B's olabel and weight in sorted order
  View dOut;  // D by (src, ilabel), with D's olabel and weight in sorted order
  const uint32_t *bflags;  // per B state: an eps:eps arc (1), a y:eps arc, y != eps (2)
  uint32_t shB, shD;
  unsigned long long *tab;
  uint32_t hmask;
  uint32_t *coacc;          // co-accessible slots (bitmap)
  const uint32_t *in_off;   // in-arcs of each slot: in_src[in_off[s] .. in_off[s + 1])
  const uint32_t *in_src;
  const int32_t *id_of;     // slot -> state id of C (-1: not trim)
};

// Units (forward) or in-arcs (backward) of a heavy key that one search
// thread of a three-input search takes.
constexpr uint32_t CHUNK3 = 8;

// A level of a three-input search in a ring of three: its frontier entries
// F[fbase, fbase + fcount) and the number of heavy-state chunks it listed.
struct Lvl3 {
  uint32_t fbase, fcount, ccount, pad;
};

// Device scalars of a three-input composition, read back by the host.
struct Scal3 {
  uint32_t errA, errB, errD, maxA, maxB, maxD;
  uint32_t overflow, levels, narcs, ntrim;
  uint32_t ncont;            // keys a search walk went on to (not in the frontier)
  uint32_t nseg;             // chain segments the forward jumps recorded
  uint32_t nheavy[2];        // heavy states of C (and an overflow word)
  unsigned long long total;  // scan totals
  Lvl3 ring[3];
};

struct Search3 {
  uint32_t *F;       // frontier slots, level after level
  uint32_t fcap;
  uint2 *chunks;     // (slot, first unit) of the chunks of heavy keys: two
  uint32_t ccap;     // lists of ccap entries (levels of even / odd number)
  uint2 *arcs;       // generated arcs (source slot, target slot)
  unsigned long long acap;
  Lvl3 *ring;
  Scal3 *sc;
  // Chain segments (optional, null to go without): a forward jump from key
  // k_0 over k_1 .. k_m records the slots of k_0 .. k_(m-1) as segment i
  // (segs[8 i .. 8 i + m)) and seg_of[slot of k_m] = i << 4 | m, so the
  // backward search claims the keys leading to k_m together.
  uint32_t *segs;
  uint32_t *seg_of;
  uint32_t scap;
};

// Output arrays of a three-input C.
struct OutGraph3 {
  int32_t *arc_offset, *src, *dst, *il, *ol;
  float *w;
  uint8_t *start, *accept;
  int32_t *key_a, *key_b;
  uint8_t *key_fab;
  int32_t *key_d;
  uint8_t *key_f;
  int32_t *arc_a, *arc_b, *arc_d;
};

// ---------------------------------------------------------------------------
// Scores of an acyclic graph (score.hip)
// ---------------------------------------------------------------------------

// The caller's graph plus its in-arc structure: inref[v] >= 0 is v's only
// in-arc, -1 means none, and -2 - m names merge m (a state with two or more
// in-arcs), whose in-arcs are marc[mbeg[m] .. mbeg[m] + mlen[m]) in any order.
struct ScoreGraph {
  int32_t V;
  long long E;
  const int32_t *off, *src, *dst;
  const float *w;
  const uint8_t *start, *accept;
  const int32_t *inref;
  const int32_t *mbeg, *mlen, *marc;
  // relaxation sweeps only (else null): the in-arcs as a CSR by target,
  // the in-arcs of v at [ioff[v], ioff[v + 1]) with their sources isrc and
  // weights iw (in no particular order)
  const int32_t *ioff, *isrc;
  const float *iw;
};

// Relaxation sweeps of a score queued between two read-backs, at most.
constexpr int SWEEP_BATCH = 64;

// Device scalars of a score computation, read back by the host.
struct ScoreScalars {
  uint32_t err, maxlab;      // validation
  uint32_t overflow, gens;   // a list overflowed; generations that had work
  uint32_t nmerge, bad;      // merges; a provenance index out of range
  unsigned long long finished;  // states given a value
  unsigned long long mtotal;    // in-arcs of all merges
  unsigned long long zmax, zlo, zhi;  // total: order key of the maximum, 128-bit sum
  uint32_t absmax, pad;         // scatter: bits of the largest |gradient|
  GenSlot G[3];
  unsigned long long rise[SWEEP_BATCH];  // sweeps: order key of each sweep's largest rise
};

// One direction of the score recursion (forward: alpha from in-arcs;
// backward: beta from out-arcs): records, term slots, values, pending counters and
// largest terms (per state), the generation lists (light states in Q,
// heavy states in H with their workgroup offsets in hoff; cap entries each),
// and the depth budget of a thread's walk.
struct ScoreArgs {
  ScoreGraph G;
  int4 *rec;     // per-state record of this direction
  double *term;  // term slots (value + weight) for pulls: 2 E entries
  const int32_t *mpos;  // position of an in-arc of a merge in marc
  unsigned long long *mkey;  // per state: order key of its largest term so far
  double *val;
  int32_t *pend;
  int32_t *Q, *H;
  uint32_t *hoff;
  uint32_t cap;
  int chain;
  ScoreScalars *sc;
};

// ---------------------------------------------------------------------------
// Keys: ((qa << shiftB | qb) << 1) | f, in canonical (qa, qb, f) order.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t make_key(uint32_t qa, uint32_t qb, uint32_t f,
                                             uint32_t shiftB) {
  return (((qa << shiftB) | qb) << 1) | f;
}
__device__ __forceinline__ uint32_t key_f(uint32_t k) { return k & 1u; }
__device__ __forceinline__ uint32_t key_qb(uint32_t k, uint32_t shiftB) {
  return (k >> 1) & ((1u << shiftB) - 1u);
}
__device__ __forceinline__ uint32_t key_qa(uint32_t k, uint32_t shiftB) {
  return (k >> 1) >> shiftB;
}
__device__ __forceinline__ bool test_bit(const uint32_t *bm, uint32_t k) {
  return (bm[k >> 5] >> (k & 31u)) & 1u;
}
// Bit of key k in the search bitmaps (diagonal layout, see Problem).
__device__ __forceinline__ uint32_t search_bit(const Problem &P, uint32_t k) {
  const uint32_t qa = key_qa(k, P.shiftB), qb = key_qb(k, P.shiftB);
  return (((qb - qa) & P.maskB) * P.rowA + qa) << 1 | (k & 1u);
}

// ---------------------------------------------------------------------------
// Wavefront / workgroup primitives
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T x) {
  const unsigned lane = __lane_id();
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    T y = __shfl_up(x, (unsigned)o, WAVE);
    if (lane >= (unsigned)o) x += y;
  }
  return x;
}

// The same for 32-bit values with DPP moves instead of LDS shuffles: adds
// of the values shifted by 1, 2, 4 and 8 lanes inside each row of 16 lanes
// (lanes shifted in from outside the row add 0), then of row 0's and row
// 2's last lane to rows 1 and 3, then of lane 31 to rows 2 and 3.
template <>
__device__ __forceinline__ uint32_t wave_incl_scan<uint32_t>(uint32_t x) {
  static_assert(WAVE == 64, "four rows of 16 lanes");
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Exclusive scan over the NT threads of a workgroup.  Every thread must call
// it (it contains barriers).  s_wsum needs NWAVES entries.
template <typename T>
__device__ __forceinline__ T block_excl_scan(T x, T *s_wsum, T &total) {
  const unsigned lane = __lane_id();
  const unsigned wid = threadIdx.x / WAVE;
  T inc = wave_incl_scan(x);
  if (lane == WAVE - 1) s_wsum[wid] = inc;
  __syncthreads();
  T off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NWAVES; ++w) {
    T s = s_wsum[w];
    if ((unsigned)w < wid) off += s;
    tot += s;
  }
  __syncthreads();
  total = tot;
  return off + inc - x;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, WAVE);
  return x;
}

// Sum over the NT threads of a workgroup, valid in thread 0.  Every thread
// must call it (it contains a barrier).
template <typename T>
__device__ __forceinline__ T block_sum(T x, T *s_w) {
  x = wave_sum(x);
  if (__lane_id() == 0) s_w[threadIdx.x / WAVE] = x;
  __syncthreads();
  T t = 0;
  if (threadIdx.x == 0)
    for (int w = 0; w < NWAVES; ++w) t += s_w[w];
  return t;
}

// First index in [lo, hi) whose value is >= x (values sorted ascending).
__device__ __forceinline__ int32_t lower_bound_i32(const int32_t *a, int32_t lo, int32_t hi,
                                                   int32_t x) {
  while (lo < hi) {
    int32_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}
// First index in [lo, hi) whose value is > x.
__device__ __forceinline__ int32_t upper_bound_i32(const int32_t *a, int32_t lo, int32_t hi,
                                                   int32_t x) {
  while (lo < hi) {
    int32_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Optional pair of HIP events that brackets one kernel launch on its stream
// (both null: no timing).
struct KernelTimer {
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  void begin(hipStream_t s) const {
    if (ev0) (void)hipEventRecord(ev0, s);
  }
  void end(hipStream_t s) const {
    if (ev1) (void)hipEventRecord(ev1, s);
  }
};

// ---------------------------------------------------------------------------
// Host-side launchers (primitives.hip)
// ---------------------------------------------------------------------------

// Bytes of temporary storage for scan_u32 over n elements.
size_t scan_temp_bytes(size_t n);
// out[i] = sum of in[0..i) (exclusive); in and out may alias.  The grand
// total (64-bit) goes to *total_dev; if out_last is true, out[n] = total
// (truncated to 32 bits).
hipError_t scan_u32(const uint32_t *in, uint32_t *out, size_t n, bool out_last,
                    unsigned long long *total_dev, void *temp, hipStream_t s);

// Bytes of temporary storage for radix_sort over n elements.
size_t sort_temp_bytes(size_t n);
// Stable LSD radix sort of (key, value) pairs on the low `bits` key bits,
// ping-ponging between (k0, v0) and (k1, v1); *in_second says whether the
// sorted result ended in (k1, v1).
hipError_t radix_sort(unsigned long long *k0, int32_t *v0, unsigned long long *k1, int32_t *v1,
                      size_t n, int bits, void *temp, hipStream_t s, bool *in_second);

// ---------------------------------------------------------------------------
// Host-side launchers (compose.hip)
// ---------------------------------------------------------------------------
// Validation of g's structure (offsets, sources, targets, flags) and, for
// side 0 (A: matched label = olabel) or 1 (B: ilabel), its labels, the
// largest matched label and whether the arcs are in label order; side 2
// checks the structure only.  *nacc (if given) += number of accepting states.
// check = false skips the checks and only gathers the label facts and nacc.
hipError_t launch_validate(const DevGraph &g, int side, uint32_t *err, uint32_t *maxlab,
                           hipStream_t s, uint32_t *nacc = nullptr, bool check = true);
// Views are built in two steps.  sort_view: sort the arcs of a view (side
// 0: A by olabel, side 1: B by ilabel; by_dst selects in-views, for which
// `off_tmp` (V+1 words) receives the group offsets; an out-view of an input
// whose groups are already in label order (presorted) is not sorted) into
// arec / perm, gather olab / w for out-views, and write the first record of
// every state.  k0/v0/k1/v1 are E-sized sort buffers.  eps_rec is A's
// out-view records when building A's in-view (to carry epsOutA), else null.
// If eps_states is set, it counts the states with an epsilon arc in the
// view.  Then finish_views (once all four views are sorted) sets FLAG_UNIQ
// (from the opposite view of the same graph), marks the arcs, writes the
// second record of every state and the label buckets.
hipError_t sort_view(const DevGraph &g, int side, bool by_dst, bool presorted, int lab_bits,
                     int4 *srec, int2 *arec, int32_t *perm, int32_t *olab, float *w,
                     int32_t *off_tmp, const int4 *eps_rec, unsigned long long *k0, int32_t *v0,
                     unsigned long long *k1, int32_t *v1, void *sort_temp, uint32_t *eps_states,
                     hipStream_t s);

// One view for finish_views: its records and arcs, the opposite view's
// (`other`), the states excluded from FLAG_UNIQ (start states for out-views,
// accepting states for in-views), the graph side (0 = A, 1 = B) and, when
// lut is set, its bucket table with lstride labels per state.
struct ViewJob {
  int4 *srec;
  int2 *arec;
  int4 *lut;
  const int4 *other;
  const int2 *other_arec;
  const uint8_t *excl;
  int32_t side, out_view, lstride;
  int4 *chain;  // chain records to write, or null
};
// Four views with the prefix sums of their state, arc and bucket counts
// (entry 4 is the total).
struct ViewJobs {
  ViewJob j[4];
  long long vbegin[5], ebegin[5], lbegin[5];
};
hipError_t finish_views(ViewJobs J, hipStream_t s);
// Collect the start states of A and B into la/lb (counts na/nb, zeroed by the
// caller) and place every start key in generation 0 of the forward search.
// Accepting keys reached by the forward search (start keys included) are
// marked co-accessible and listed in S.acc (count in Scalars::tail2).
hipError_t launch_seed_forward(const Problem &P, const SearchArgs &S, int32_t *la, uint32_t *na,
                               int32_t *lb, uint32_t *nb, hipStream_t s);
// Collect the accepting states of A and B into la/lb (counts na/nb, zeroed
// by the caller) and place every accepting key (f = 0, and f = 1 where
// epsOutA) in generation 0 of a backward search over all key pairs.
hipError_t launch_seed_backward_all(const Problem &P, const SearchArgs &S, int32_t *la,
                                    uint32_t *na, int32_t *lb, uint32_t *nb, hipStream_t s);
// Place the accepting keys listed by the forward search (acc_list) in
// generation 0 of the backward search.
hipError_t launch_seed_backward(const Problem &P, const SearchArgs &S, const uint32_t *acc_list,
                                hipStream_t s);
// Generation g of the forward (or backward) search: one kernel.
hipError_t launch_generation(const Problem &P, const SearchArgs &S, bool forward, int g,
                             hipStream_t s);
// Generation gf of a forward search (SF) and generation gb of a backward
// search (SB) running side by side in one kernel (half of the workgroups
// each).
hipError_t launch_generation2(const Problem &P, const SearchArgs &SF, const SearchArgs &SB, int gf,
                              int gb, hipStream_t s);
// *out += number of moves the forward search examines out of the keys set in
// P.vis (search layout, nwords words), or (backward) the backward search
// examines into the keys set in P.trim (key order, nwords words): a
// statistic.
hipError_t launch_count_moves(const Problem &P, size_t nwords, bool forward,
                              unsigned long long *out, hipStream_t s);
// *out += number of set bits of bm[0, nwords).
hipError_t launch_popcount(const uint32_t *bm, size_t nwords, unsigned long long *out,
                           hipStream_t s);
// The trim bitmap in key order from the two search bitmaps (search layout):
// trim = vis AND coacc, transposed from diagonals to rows of A states, and
// cnt[w] = popcount(trim[w]) for each of its VA << (shiftB + 1) / 32 words.
// Needs shiftB >= 4 (a trim word then holds keys of one A state).
hipError_t launch_trim(const Problem &P, uint32_t VA, uint32_t *trim, uint32_t *cnt,
                       hipStream_t s);
// Kept-arc count of every state of C, one chunk of OUT_WORDS trim words per
// wavefront: cnt8[id] (255: the count is in cnt32[id]) for light states,
// heavy states listed in `heavy` as (id, key) (their number in
// Scalars::heavy), btot[chunk] = the chunk's light total.
hipError_t launch_count(const Problem &P, size_t nwords, uint8_t *cnt8, uint32_t *cnt32,
                        uint32_t *btot, uint2 *heavy, Scalars *sc, hipStream_t s);
// Counts of the heavy states (cnt8 / cnt32, added to their chunk's btot).
hipError_t launch_count_heavy(const Problem &P, const uint2 *heavy, const uint32_t *nheavy_dev,
                              uint8_t *cnt8, uint32_t *cnt32, uint32_t *btot, hipStream_t s);
// Write C: btot holds the exclusive arc offset of every chunk.
hipError_t launch_fill(const Problem &P, size_t nwords, const uint8_t *cnt8,
                       const uint32_t *cnt32, const uint32_t *btot, const uint2 *heavy,
                       uint32_t nheavy, uint32_t nstates, uint32_t narcs, const OutGraph &O,
                       hipStream_t s);

// Batches (compose.hip): copy item graph a into the union arrays at state
// offset vbase and arc offset ebase (off, src, dst shifted); and, after a
// run on the union, the first state and first arc of every item (out[i],
// out[n + 1 + i] for i <= n; qa_base[i] = the item's first state of A).
hipError_t launch_union_copy(const DevGraph &a, long long vbase, long long ebase, int32_t *off,
                             int32_t *src, int32_t *dst, hipStream_t s);
hipError_t launch_item_ranges(const Problem &P, unsigned long long nkeys, int32_t n,
                              const long long *qa_base, const uint8_t *cnt8,
                              const uint32_t *cnt32, const uint32_t *btot, uint32_t nstates,
                              uint32_t narcs, long long *out, hipStream_t s);

// Three-input launchers (compose3.hip).
hipError_t launch3_bflags(const DevGraph &B, uint32_t *bflags, hipStream_t s);
// Bucket table of a view (v.lut with v.lstride labels per state) from its
// records and arcs.
hipError_t launch3_lut(const View &v, long long nstates, hipStream_t s);
// Chain records (CHAIN_INT4 int4 per state) of B's out-view for the chain
// jumps of the forward search.
hipError_t launch3_chains(const View &v, long long nstates, int4 *chain, hipStream_t s);
// Start keys of every triple of start states (lists and counts from
// launch3_starts) into level 0 of S.
hipError_t launch3_starts(const DevGraph &A, const DevGraph &B, const DevGraph &D,
                          int32_t *lists, uint32_t *counts, hipStream_t s);
hipError_t launch3_seed(const Problem3 &P, const Search3 &S, const int32_t *lists,
                        const uint32_t *counts, hipStream_t s);
// Level l of the forward (or backward) search: two kernels.
hipError_t launch3_level(const Problem3 &P, const Search3 &S, bool forward, int l,
                         hipStream_t s);
// The generated arcs as (target, source) pairs for a sort by target; then,
// over the sorted targets, every target's in-degree (indeg, zeroed by the
// caller; first: H scratch entries).
hipError_t launch3_arc_keys(const uint2 *arcs, unsigned long long narcs, unsigned long long *key,
                            int32_t *src, hipStream_t s);
hipError_t launch3_in_degrees(const unsigned long long *key, unsigned long long narcs,
                              uint32_t *first, uint32_t *indeg, hipStream_t s);
hipError_t launch3_seed_bwd(const Problem3 &P, const Search3 &S, hipStream_t s);
hipError_t launch3_collect(const Problem3 &P, unsigned long long *keys, int32_t *slots,
                           uint32_t *count, uint32_t cap, uint32_t *overflow, hipStream_t s);
// id_of (slot -> state id), units per state, heavy states (more units
// than one thread takes; count in nheavy[0], nheavy[1] an overflow word).
hipError_t launch3_ids(const Problem3 &P, const unsigned long long *keys, const int32_t *slots,
                       uint32_t n, int32_t *id_of, uint32_t *units, uint32_t *heavy,
                       uint32_t *nheavy, hipStream_t s);
// Kept arcs per work unit (ustart: n + 1 unit offsets per state).
hipError_t launch3_count(const Problem3 &P, const unsigned long long *keys,
                         const uint32_t *ustart, uint32_t n, const uint32_t *heavy,
                         const uint32_t *nheavy, uint32_t *ucnt, hipStream_t s);
// Write C (uoff: U + 1 arc offsets per unit).
hipError_t launch3_fill(const Problem3 &P, const unsigned long long *keys, const uint32_t *ustart,
                        uint32_t n, const uint32_t *heavy, const uint32_t *nheavy,
                        const uint32_t *uoff, uint32_t narcs, const OutGraph3 &O,
                        hipStream_t s);

// Score launchers (score.hip).
// In-arc structure of G: owner (V words, all -1) and extra (V words, all 0)
// are scratch; inref (V), mbeg/mlen/mcur (V each), marc (E) and mpos (E;
// set for the in-arcs of merges) receive it; sc->nmerge and sc->mtotal
// must be 0.
hipError_t launch_score_structure(const ScoreGraph &G, int32_t *owner, int32_t *extra,
                                  int32_t *inref, int32_t *mbeg, int32_t *mlen, int32_t *mcur,
                                  int32_t *marc, int32_t *mpos, ScoreScalars *sc,
                                  hipStream_t s);
// Pending counters and generation 0 of one direction (sc->G zeroed).
hipError_t launch_score_seed(const ScoreArgs &S, bool forward, hipStream_t s);
// Generation g of the forward (F) and / or backward (B) recursion: one kernel.
hipError_t launch_score_generation(const ScoreArgs *F, const ScoreArgs *B, int g,
                                   hipStream_t s);
// One relaxation sweep of the score recursions (graphs with cycles): ya[v]
// = forward value of v from the previous values xa, yb[v] = backward value
// from xb (a null output skips that direction; G needs the in-arc
// structure); *incr = max(*incr, order key of the largest rise of a value).
hipError_t launch_sweep(const ScoreGraph &G, const double *xa, double *ya, const double *xb,
                        double *yb, unsigned long long *incr, hipStream_t s);
// p[0 .. n) = x.
hipError_t launch_fill_f64(double *p, long long n, double x, hipStream_t s);
// The in-arc CSR of G for the sweeps (counting by target, a scan, then
// each arc placed with an atomic cursor): ioff (V + 1 words), isrc and iw (E
// each), cur (V words of scratch); scan_temp of scan_temp_bytes(V) bytes.
hipError_t launch_in_csr(const ScoreGraph &G, int32_t *ioff, int32_t *isrc, float *iw,
                         int32_t *cur, void *scan_temp, unsigned long long *total_dev,
                         hipStream_t s);
// *total = log-add of val[v] over the states with flag[v] (sc->zmax, zlo,
// zhi zeroed).
hipError_t launch_score_total(const double *val, const uint8_t *flag, int32_t V,
                              ScoreScalars *sc, double *total, hipStream_t s);
// totals[i] = log-add of val[v] over the flagged v in [bounds[i],
// bounds[i + 1]) for i < n (bounds: n + 1 device words; max_len the longest
// segment; z: 3 n words, zeroed by the caller).
hipError_t launch_segment_logsum(const double *val, const uint8_t *flag, int32_t n,
                                 const long long *bounds, long long max_len,
                                 unsigned long long *z, double *totals, hipStream_t s);
// grad[e] = scale * exp(alpha[src e] + w(e) + beta[dst e] - *total).
hipError_t launch_posterior(const ScoreGraph &G, const double *alpha, const double *beta,
                            const double *total, float scale, float *grad, hipStream_t s);
// Workspace of the grouped scatter: the terms grouped by target range (pg,
// pidx: n each), the per-workgroup bucket counts (scatter_count_words), scan
// storage for them and the number of grouped terms.
struct ScatterTemp {
  float *pg;
  int32_t *pidx;
  uint32_t *cnt;
  void *scan;
  unsigned long long *total;
};
// Whether launch_scatter groups the terms first (when given a ScatterTemp).
bool scatter_grouped(long long n, int32_t m);
size_t scatter_count_words(long long n, int32_t m);
// out[i] = sum of g[e] over e < n with idx[e] = i; acc (4 m words), *mx and
// *bad zeroed by the caller; *bad becomes nonzero if an index is out of range.
// With tmp (may be null) the terms are grouped by target range first when
// scatter_grouped(n, m).
hipError_t launch_scatter(const float *g, const int32_t *idx, long long n, int32_t m,
                          unsigned long long *acc, uint32_t *mx, uint32_t *bad, float *out,
                          const ScatterTemp *tmp, hipStream_t s);
// The address, on `device` (which must be current), of the device array
// that fst_grad_scatter_noalloc works in; looked up once per device.
hipError_t scatter_scratch(int device, void **out);
// launch_scatter without grouping, with its accumulators and scalars in
// that array (scr, from scatter_scratch): clears what the call uses, then
// sums; m <= FST_SCATTER_NOALLOC_MAX_TARGETS.  The bad-index flag is 32-bit
// word 1 of scr.
hipError_t launch_scatter_noalloc(const float *g, const int32_t *idx, long long n, int32_t m,
                                  void *scr, float *out, hipStream_t s);

}  // namespace fstc
