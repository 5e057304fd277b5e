// Device-wide primitives for gfx950: exclusive scan and a stable LSD radix
// sort.  Both are tiled for 256-thread workgroups of four 64-wide wavefronts
// with coalesced loads (consecutive threads touch consecutive words).
#include "internal.h"

namespace fstc {

namespace {

constexpr int SCAN_ITEMS = 8;
constexpr size_t SCAN_TILE = (size_t)NT * SCAN_ITEMS;
// Elements per thread of a sort tile: small inputs (the views of most
// operands) take short tiles for more workgroups, large ones long tiles for a
// smaller digit histogram.
inline int sort_items(size_t n) { return n <= ((size_t)1 << 20) ? 4 : 16; }
constexpr uint32_t SORT_LOCAL = 256;  // tiles up to which a pass needs no scan

typedef unsigned long long ull;

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

template <typename TI>
__global__ __launch_bounds__(NT) void k_scan_reduce(const TI *__restrict__ in, size_t n,
                                                    ull *__restrict__ part) {
  __shared__ ull s_w[NWAVES];
  const size_t base = (size_t)blockIdx.x * SCAN_TILE;
  ull s = 0;
#pragma unroll
  for (int r = 0; r < SCAN_ITEMS; ++r) {
    size_t i = base + (size_t)r * NT + threadIdx.x;
    if (i < n) s += (ull)in[i];
  }
  s = wave_sum(s);
  if (__lane_id() == 0) s_w[threadIdx.x / WAVE] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    ull t = 0;
    for (int w = 0; w < NWAVES; ++w) t += s_w[w];
    part[blockIdx.x] = t;
  }
}

template <typename TI, typename TO>
__global__ __launch_bounds__(NT) void k_scan_final(const TI *in, TO *out, size_t n,
                                                   const ull *__restrict__ part_scanned,
                                                   ull *__restrict__ total, int out_last) {
  __shared__ ull s_w[NWAVES];
  const size_t base = (size_t)blockIdx.x * SCAN_TILE;
  ull carry = part_scanned ? part_scanned[blockIdx.x] : 0ull;
  for (int r = 0; r < SCAN_ITEMS; ++r) {
    size_t i = base + (size_t)r * NT + threadIdx.x;
    ull x = (i < n) ? (ull)in[i] : 0ull;
    ull tot;
    ull ex = block_excl_scan<ull>(x, s_w, tot);
    if (i < n) out[i] = (TO)(carry + ex);
    carry += tot;
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    *total = carry;
    if (out_last) out[n] = (TO)carry;
  }
}

// Temp layout for a scan over n: [block sums (nb ull)] [temp of their scan].
size_t scan_temp_rec(size_t n) {
  size_t nb = (n + SCAN_TILE - 1) / SCAN_TILE;
  if (nb <= 1) return 0;
  return align_up(nb * sizeof(ull)) + scan_temp_rec(nb);
}

template <typename TI, typename TO>
hipError_t scan_rec(const TI *in, TO *out, size_t n, bool out_last, ull *total, char *temp,
                    hipStream_t s) {
  size_t nb = (n + SCAN_TILE - 1) / SCAN_TILE;
  if (nb <= 1) {
    k_scan_final<TI, TO><<<1, NT, 0, s>>>(in, out, n, nullptr, total, out_last ? 1 : 0);
    return hipGetLastError();
  }
  ull *part = reinterpret_cast<ull *>(temp);
  char *rest = temp + align_up(nb * sizeof(ull));
  k_scan_reduce<TI><<<(unsigned)nb, NT, 0, s>>>(in, n, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Scan the block sums in place.  Their grand total is written to *total,
  // which the final pass below overwrites (stream order) with the real one.
  e = scan_rec<ull, ull>(part, part, nb, false, total, rest, s);
  if (e != hipSuccess) return e;
  k_scan_final<TI, TO><<<(unsigned)nb, NT, 0, s>>>(in, out, n, part, total, out_last ? 1 : 0);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// radix sort
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) void k_radix_hist(const ull *__restrict__ k, size_t n,
                                                   int shift, uint32_t *__restrict__ hist,
                                                   uint32_t nb, int items) {
  __shared__ uint32_t s_h[256];
  s_h[threadIdx.x] = 0;
  __syncthreads();
  const size_t base = (size_t)blockIdx.x * NT * items;
#pragma unroll 4
  for (int r = 0; r < items; ++r) {
    size_t i = base + (size_t)r * NT + threadIdx.x;
    if (i < n) atomicAdd(&s_h[(uint32_t)(k[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  hist[(size_t)threadIdx.x * nb + blockIdx.x] = s_h[threadIdx.x];
}

// Stable scatter: inside the tile, elements are ranked in index order.  Each
// round ranks 256 elements: inside a wavefront by matching the 8 digit bits
// with ballots, across the four wavefronts through LDS counts.  With
// local_offsets the histogram is the raw per-tile counts (digit-major, at
// most SORT_LOCAL tiles) and every workgroup forms its own starting offsets
// (thread d: digit d's counts over all tiles and over the tiles before its
// own, then a workgroup scan over the digits), which saves the device-wide
// scan of small sorts.
__global__ __launch_bounds__(NT) void k_radix_scatter(const ull *__restrict__ kin,
                                                      const int32_t *__restrict__ vin,
                                                      ull *__restrict__ kout,
                                                      int32_t *__restrict__ vout, size_t n,
                                                      int shift,
                                                      const uint32_t *__restrict__ gofs,
                                                      uint32_t nb, int items, int local_offsets) {
  __shared__ uint32_t s_run[256];
  __shared__ uint32_t s_wc[NWAVES][256];
  const unsigned tid = threadIdx.x, wid = tid / WAVE;
  if (local_offsets) {
    uint32_t total = 0, before = 0;
    const uint32_t *h = gofs + (size_t)tid * nb;
#pragma unroll 16
    for (uint32_t t = 0; t < nb; ++t) {
      const uint32_t c = h[t];
      total += c;
      before += t < blockIdx.x ? c : 0u;
    }
    __shared__ uint32_t s_sum[NWAVES];
    uint32_t all;
    s_run[tid] = block_excl_scan<uint32_t>(total, s_sum, all) + before;
  } else {
    s_run[tid] = gofs[(size_t)tid * nb + blockIdx.x];
  }
  const size_t base = (size_t)blockIdx.x * NT * items;
  // each round loads the next round's key and value before its own work
  ull key_next = 0ull;
  int32_t val_next = 0;
  if (base + tid < n) {
    key_next = kin[base + tid];
    val_next = vin[base + tid];
  }
  for (int r = 0; r < items; ++r) {
#pragma unroll
    for (int w = 0; w < NWAVES; ++w) s_wc[w][tid] = 0;
    const size_t i = base + (size_t)r * NT + tid;
    const bool valid = i < n;
    const ull key = key_next;
    const int32_t val = val_next;
    if (r + 1 < items && i + NT < n) {
      key_next = kin[i + NT];
      val_next = vin[i + NT];
    }
    __syncthreads();
    uint32_t d = (uint32_t)(key >> shift) & 255u;
    unsigned long long m = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      unsigned long long bb = __ballot((d >> b) & 1u);
      m &= ((d >> b) & 1u) ? bb : ~bb;
    }
    uint32_t rank = (uint32_t)__popcll(m & __lanemask_lt());
    if (valid && rank == 0) s_wc[wid][d] = (uint32_t)__popcll(m);
    __syncthreads();
    if (valid) {
      uint32_t pos = s_run[d] + rank;
      for (unsigned w = 0; w < wid; ++w) pos += s_wc[w][d];
      kout[pos] = key;
      vout[pos] = val;
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int w = 0; w < NWAVES; ++w) add += s_wc[w][tid];
    s_run[tid] += add;
    __syncthreads();
  }
}

}  // namespace

size_t scan_temp_bytes(size_t n) { return scan_temp_rec(n) + 256; }

hipError_t scan_u32(const uint32_t *in, uint32_t *out, size_t n, bool out_last,
                    unsigned long long *total_dev, void *temp, hipStream_t s) {
  return scan_rec<uint32_t, uint32_t>(in, out, n, out_last, total_dev,
                                      reinterpret_cast<char *>(temp), s);
}

// Enough for every radix_sort of at most n elements (the tile depends on the
// element count).
size_t sort_temp_bytes(size_t n) {
  const size_t small = n < ((size_t)1 << 20) ? n : ((size_t)1 << 20);
  const size_t ts = (size_t)NT * sort_items(small), tl = (size_t)NT * sort_items(n + 1);
  const size_t nbs = (small + ts - 1) / ts, nbl = (n + tl - 1) / tl;
  const size_t nb = nbs > nbl ? nbs : nbl;
  size_t nh = 256 * (nb ? nb : 1);
  return align_up(nh * sizeof(uint32_t)) + align_up(sizeof(ull)) + scan_temp_bytes(nh);
}

hipError_t radix_sort(unsigned long long *k0, int32_t *v0, unsigned long long *k1, int32_t *v1,
                      size_t n, int bits, void *temp, hipStream_t s, bool *in_second) {
  *in_second = false;
  if (n == 0 || bits <= 0) return hipSuccess;
  const int items = sort_items(n);
  const size_t tile = (size_t)NT * items;
  const uint32_t nb = (uint32_t)((n + tile - 1) / tile);
  const size_t nh = (size_t)256 * nb;
  char *t = reinterpret_cast<char *>(temp);
  uint32_t *hist = reinterpret_cast<uint32_t *>(t);
  ull *tot = reinterpret_cast<ull *>(t + align_up(nh * sizeof(uint32_t)));
  void *stemp = t + align_up(nh * sizeof(uint32_t)) + align_up(sizeof(ull));
  ull *ka = k0, *kb = k1;
  int32_t *va = v0, *vb = v1;
  int passes = (bits + 7) / 8;
  for (int p = 0; p < passes; ++p) {
    int shift = 8 * p;
    k_radix_hist<<<nb, NT, 0, s>>>(ka, n, shift, hist, nb, items);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int local = nb <= SORT_LOCAL ? 1 : 0;
    if (!local) {
      e = scan_u32(hist, hist, nh, false, tot, stemp, s);
      if (e != hipSuccess) return e;
    }
    k_radix_scatter<<<nb, NT, 0, s>>>(ka, va, kb, vb, n, shift, hist, nb, items, local);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    ull *tk = ka; ka = kb; kb = tk;
    int32_t *tv = va; va = vb; vb = tv;
  }
  *in_second = ka != k0;
  return hipSuccess;
}

}  // namespace fstc
