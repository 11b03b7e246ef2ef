// Graph layout on the GPU: CSR validation, in/out degrees, degree-sorted row
// order (stable LSD radix sort, largest degree first), row segments of at
// most seg_len edges and row blocks of bounded cost.
//
// The degree skew of real graphs follows a power law (Sec. 3.2, Fig. 8a of
// the paper); batching vertices by degree as the profiled library did left
// the GPU idle (Fig. 8b/c).  Here the sorted order only schedules work: rows
// of similar degree share a workgroup, the heaviest rows start first, and a
// row longer than seg_len is split across several lanes groups so that no
// single wave walks a hub row alone.
#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 8;
constexpr int kTile = kThreads * kItems;  // 2048 items per workgroup tile
constexpr int kBins = 256;                // 8-bit radix digits

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// ------------------------------------------------------------------------
// block-wide scans (blockDim.x == NT)
// ------------------------------------------------------------------------
__device__ __forceinline__ int32_t wave_incl_scan(int32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int32_t y = __shfl_up(v, off, 64);
    if (lane >= off) v += y;
  }
  return v;
}

template <int NT>
__device__ __forceinline__ int32_t block_excl_scan(int32_t v, int32_t* total) {
  __shared__ int32_t ws[NT / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int32_t incl = wave_incl_scan(v);
  if (lane == 63) ws[wave] = incl;
  __syncthreads();
  int32_t off = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < NT / 64; ++k) {
    if (k < wave) off += ws[k];
    tot += ws[k];
  }
  __syncthreads();
  *total = tot;
  return off + incl - v;
}

// ------------------------------------------------------------------------
// functors feeding the generic scan
// ------------------------------------------------------------------------
struct ArrF {
  const int32_t* p;
  __device__ int32_t operator()(int64_t i) const { return p[i]; }
};
// the in-degree behind a degree-order sort key (key = 0x7fffffff - d_in)
__device__ __forceinline__ int32_t key_degree(uint32_t key) { return (int32_t)(0x7fffffffu - key); }
// number of segments of perm position i, from the sorted keys
struct NsegF {
  const uint32_t* keys;
  int32_t T;
  __device__ int32_t operator()(int64_t i) const {
    const int32_t d = key_degree(keys[i]);
    return d > T ? (d + T - 1) / T : 1;
  }
};
// cost of segment s
struct CostF {
  const int32_t* beg;
  const int32_t* end;
  int32_t c;
  __device__ int32_t operator()(int64_t i) const { return end[i] - beg[i] + c; }
};

// ------------------------------------------------------------------------
// kernels
// ------------------------------------------------------------------------
__global__ void k_zero(int32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// d_in, d_out and CSR validation; error bits go to counts[kErrFlags]
// (edges_too: also count d_out with global atomics -- only used when the
// source range is too large for the bucketed count below)
__global__ __launch_bounds__(kThreads) void k_degrees(const int32_t* __restrict__ rp,
                                                      const int32_t* __restrict__ col, int32_t V,
                                                      int32_t Vs, int64_t E, int edges_too,
                                                      int32_t* d_in, int32_t* d_out,
                                                      int32_t* counts) {
  int err = 0;
  int maxd = 0;
  const int64_t n = (V > E || !edges_too) ? (int64_t)V : E;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < V) {
      int32_t a = rp[i], b = rp[i + 1];
      if (b < a) err |= 2;
      int32_t d = b - a;
      d = d < 0 ? 0 : d;
      d_in[i] = d;
      maxd = d > maxd ? d : maxd;
      if (i == 0) {
        if (a != 0) err |= 1;
        if ((int64_t)rp[V] != E) err |= 4;
      }
    }
    if (edges_too && i < E) {
      int32_t c = col[i];
      if (c < 0 || c >= Vs)
        err |= 8;
      else
        atomicAdd(&d_out[c], 1);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    err |= __shfl_xor(err, off, 64);
    int m = __shfl_xor(maxd, off, 64);
    maxd = m > maxd ? m : maxd;
  }
  // one atomic per workgroup (same-address atomics serialize)
  __shared__ int s_err[kThreads / 64], s_max[kThreads / 64];
  if ((threadIdx.x & 63) == 0) {
    s_err[threadIdx.x >> 6] = err;
    s_max[threadIdx.x >> 6] = maxd;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kThreads / 64; ++k) {
      err |= s_err[k];
      maxd = s_max[k] > maxd ? s_max[k] : maxd;
    }
    if (err) atomicOr(&counts[kErrFlags], err);
    // most workgroups already see a larger maximum: skip their atomic
    if (maxd > __hip_atomic_load(&counts[kMaxDegree], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
      atomicMax(&counts[kMaxDegree], maxd);
  }
}

// ------------------------------------------------------------------------
// Out-degrees without global atomics.  A power-law graph sends a large share
// of all edges to a few hub sources, and same-address atomics serialize, so
// instead: (1) histogram the CSR source ids by bucket (8192 ids per bucket)
// per tile, (2) scan, (3) scatter the ids into bucket order as 16-bit
// offsets within their bucket, (4) count each bucket in a 32 KB LDS
// histogram and store the counts.
// ------------------------------------------------------------------------
// Tile of this workgroup in an XCD-blocked order.  Workgroups are handed to
// the eight XCDs in turn (w % 8), so with tile = w the tiles one L2 sees are
// eight apart, and the tile-minor histogram entries of neighbouring tiles
// (32 to a 128-byte line) are written and read as partial lines through
// eight different L2s.  Here XCD x takes the contiguous run
// [x * per, (x + 1) * per) of tiles.  The grid is xcd_grid(ntiles)
// workgroups; the spare ones get -1.  Any dispatch order gives the same
// result; only the locality depends on it.
constexpr int kXcds = 8;
__device__ __forceinline__ int64_t xcd_tile(int64_t ntiles) {
  const int64_t per = (ntiles + kXcds - 1) / kXcds;
  const int64_t w = blockIdx.x, t = (w % kXcds) * per + w / kXcds;
  return t < ntiles ? t : -1;
}
inline unsigned xcd_grid(int64_t ntiles) {
  return (unsigned)(kXcds * ((ntiles + kXcds - 1) / kXcds));
}

constexpr int kBucketBits = 13;
constexpr int kBucketSize = 1 << kBucketBits;
constexpr int kMaxBuckets = 2048;  // keeps the scatter's LDS within 64 KB
constexpr int kEdgeItems = 32;
constexpr int kEdgeTile = kThreads * kEdgeItems;  // 8192 edges per tile

// per-tile bucket histogram; each wave counts into its own copy (fewer
// same-address LDS atomics), the copies are summed at the end
__global__ __launch_bounds__(kThreads) void k_outdeg_hist(const int32_t* __restrict__ col,
                                                          int64_t E, int32_t Vs, int nb,
                                                          int32_t* __restrict__ hist,
                                                          int64_t ntiles, int32_t* counts) {
  extern __shared__ int32_t h[];  // [kThreads / 64][nb]
  constexpr int NW = kThreads / 64;
  const int64_t tile = xcd_tile(ntiles);
  if (tile < 0) return;
  for (int b = threadIdx.x; b < NW * nb; b += kThreads) h[b] = 0;
  __syncthreads();
  int32_t* hw = h + (threadIdx.x >> 6) * nb;
  int err = 0;
  const int64_t base = tile * (int64_t)kEdgeTile;
  int32_t c[kEdgeItems];
#pragma unroll
  for (int j = 0; j < kEdgeItems; ++j) {
    const int64_t i = base + j * kThreads + threadIdx.x;
    c[j] = i < E ? __builtin_nontemporal_load(col + i) : -1;
  }
#pragma unroll
  for (int j = 0; j < kEdgeItems; ++j) {
    const int64_t i = base + j * kThreads + threadIdx.x;
    if (i < E) {
      if (c[j] < 0 || c[j] >= Vs)
        err |= 8;
      else
        atomicAdd(&hw[c[j] >> kBucketBits], 1);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) err |= __shfl_xor(err, off, 64);
  if ((threadIdx.x & 63) == 0 && err) atomicOr(&counts[kErrFlags], err);
  __syncthreads();
  for (int b = threadIdx.x; b < nb; b += kThreads) {
    int32_t t = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) t += h[w * nb + b];
    hist[(int64_t)b * ntiles + tile] = t;
  }
}

// Scatter one tile into bucket order.  The tile is first ranked by bucket in
// LDS, then written out so that consecutive threads store consecutive
// positions of one bucket (coalesced 16-bit stores).  `offs` is the
// exclusive scan of hist in bucket-major order, so the tile's count in
// bucket b is offs[b * ntiles + tile + 1] - offs[b * ntiles + tile].
__global__ __launch_bounds__(kThreads) void k_outdeg_scatter(const int32_t* __restrict__ col,
                                                             int64_t E, int nb,
                                                             const int32_t* __restrict__ offs,
                                                             int64_t ntiles,
                                                             uint16_t* __restrict__ out,
                                                             int32_t* counts) {
  if (counts[kErrFlags]) return;
  extern __shared__ int32_t sm[];
  __shared__ int s_bad;
  int32_t* gbase = sm;            // [nb] global start of this tile's run in bucket b
  int32_t* lbase = sm + nb;       // [nb] local start of bucket b within the tile
  int32_t* cur = sm + 2 * nb;     // [nb] local cursor
  uint16_t* sval = reinterpret_cast<uint16_t*>(sm + 3 * nb);  // [kEdgeTile]
  uint16_t* sbkt = sval + kEdgeTile;                           // [kEdgeTile]
  const int64_t tile = xcd_tile(ntiles);
  if (tile < 0) return;
  const int64_t base = tile * (int64_t)kEdgeTile;
  const int n = (int)(E - base < kEdgeTile ? E - base : kEdgeTile);
  for (int b = threadIdx.x; b < nb; b += kThreads) {
    const int64_t f = (int64_t)b * ntiles + tile;
    const int32_t g0 = offs[f];
    const int32_t g1 = f + 1 < (int64_t)nb * ntiles ? offs[f + 1] : (int32_t)E;
    gbase[b] = g0;
    cur[b] = g1 - g0;  // count, scanned below
  }
  __syncthreads();
  {  // exclusive scan of the tile's bucket counts: thread t owns buckets
     // [t * per, (t + 1) * per), then a wave scan and a cross-wave pass
    __shared__ int32_t wsum[kThreads / 64];
    const int per = (nb + kThreads - 1) / kThreads;
    const int b0 = threadIdx.x * per;
    int32_t own = 0;
    for (int k = 0; k < per; ++k)
      if (b0 + k < nb) own += cur[b0 + k];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t inc = own;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t y = __shfl_up(inc, off, 64);
      if (lane >= off) inc += y;
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int32_t run = inc - own;
    for (int w = 0; w < wave; ++w) run += wsum[w];
    int32_t total = 0;
    for (int w = 0; w < kThreads / 64; ++w) total += wsum[w];
    for (int k = 0; k < per; ++k)
      if (b0 + k < nb) {
        const int32_t c = cur[b0 + k];
        lbase[b0 + k] = run;
        cur[b0 + k] = run;
        run += c;
      }
    if (threadIdx.x == 0) {
      s_bad = total != n;
      if (s_bad) atomicOr(&counts[kErrFlags], kErrInternal);
    }
  }
  __syncthreads();
  if (s_bad) return;
  int32_t c[kEdgeItems];
#pragma unroll
  for (int j = 0; j < kEdgeItems; ++j) {
    const int64_t i = base + j * kThreads + threadIdx.x;
    c[j] = i < E ? __builtin_nontemporal_load(col + i) : 0;
  }
#pragma unroll
  for (int j = 0; j < kEdgeItems; ++j) {
    if (j * kThreads + (int)threadIdx.x < n) {
      const int b = c[j] >> kBucketBits;
      const int32_t p = atomicAdd(&cur[b], 1);
      if (p >= 0 && p < n) {
        sval[p] = (uint16_t)(c[j] & (kBucketSize - 1));
        sbkt[p] = (uint16_t)b;
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += kThreads) {
    const int b = sbkt[i];
    const int64_t g = (int64_t)gbase[b] + (i - lbase[b]);
    if (g >= 0 && g < E)
      out[g] = sval[i];
    else
      atomicOr(&counts[kErrFlags], kErrInternal);
  }
}

// kOutdegSplit workgroups per bucket, each counting one slice of the
// bucket into LDS and storing its partial histogram (a hub's occurrences are
// split over the workgroups, so same-address LDS atomics stay few per CU)
constexpr int kOutdegSplit = 8;

__global__ __launch_bounds__(1024) void k_outdeg_count(const uint16_t* __restrict__ bucketed,
                                                       const int32_t* __restrict__ offs,
                                                       int64_t ntiles, int nb, int64_t E,
                                                       int32_t Vs, int32_t* __restrict__ part,
                                                       const int32_t* counts) {
  if (counts[kErrFlags]) return;
  __shared__ int32_t h[kBucketSize];
  const int b = blockIdx.y, w = blockIdx.x;
  for (int i = threadIdx.x; i < kBucketSize; i += 1024) h[i] = 0;
  __syncthreads();
  int64_t lo = offs[(int64_t)b * ntiles];
  int64_t hi = b + 1 < nb ? (int64_t)offs[(int64_t)(b + 1) * ntiles] : E;
  lo = lo < 0 ? 0 : (lo > E ? E : lo);
  hi = hi < lo ? lo : (hi > E ? E : hi);
  const int64_t n = hi - lo;
  const int64_t s0 = lo + n * w / kOutdegSplit, s1 = lo + n * (w + 1) / kOutdegSplit;
  constexpr int kB = 8;  // loads in flight per thread before the LDS atomics
  for (int64_t i0 = s0; i0 < s1; i0 += 1024 * kB) {
    int32_t v[kB];
#pragma unroll
    for (int j = 0; j < kB; ++j) {
      const int64_t i = i0 + j * 1024 + threadIdx.x;
      v[j] = i < s1 ? (int32_t)__builtin_nontemporal_load(bucketed + i) : -1;
    }
#pragma unroll
    for (int j = 0; j < kB; ++j)
      if (v[j] >= 0) atomicAdd(&h[v[j] & (kBucketSize - 1)], 1);
  }
  __syncthreads();
  const int64_t v0 = (int64_t)b << kBucketBits;
  int32_t* pw = part + (int64_t)w * nb * kBucketSize + v0;
  for (int i = threadIdx.x; i < kBucketSize; i += 1024) pw[i] = h[i];
}

__global__ __launch_bounds__(kThreads) void k_outdeg_reduce(const int32_t* __restrict__ part,
                                                            int nb, int32_t Vs,
                                                            int32_t* __restrict__ d_out,
                                                            const int32_t* counts) {
  if (counts[kErrFlags]) return;
  const int64_t stride = (int64_t)nb * kBucketSize;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < Vs;
       v += (int64_t)gridDim.x * blockDim.x) {
    int32_t s = 0;
#pragma unroll
    for (int w = 0; w < kOutdegSplit; ++w) s += part[w * stride + v];
    d_out[v] = s;
  }
}

// per-tile digit histogram, stored digit-major: hist[digit * ntiles + tile]
template <bool FIRST>
__global__ __launch_bounds__(kThreads) void k_radix_hist(const int32_t* __restrict__ d_in,
                                                         const uint32_t* __restrict__ keys,
                                                         int32_t n, int shift,
                                                         int32_t* __restrict__ hist, int64_t ntiles,
                                                         const int32_t* counts) {
  if (counts[kErrFlags]) return;
  __shared__ int32_t h[kBins];
  const int64_t tile = xcd_tile(ntiles);
  if (tile < 0) return;
  h[threadIdx.x] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    int64_t i = tile * kTile + j * kThreads + threadIdx.x;
    if (i < n) {
      uint32_t k = FIRST ? (0x7fffffffu - (uint32_t)d_in[i]) : keys[i];
      atomicAdd(&h[(k >> shift) & (kBins - 1)], 1);
    }
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * ntiles + tile] = h[threadIdx.x];
}

// Stable scatter.  Items are visited in index order (round j, thread t ->
// item j*256 + t); an item's rank among equal digits inside the tile comes
// from a wave-level match (8 ballots) plus the counts of lower waves and of
// earlier rounds, so equal keys keep their input order.
// Each item carries a second value, its row's first CSR entry (row_ptr[v]
// on the first pass), so that the segment builder reads it in perm order
// instead of gathering row_ptr at random.
template <bool FIRST>
__global__ __launch_bounds__(kThreads) void k_radix_scatter(
    const int32_t* __restrict__ d_in, const uint32_t* __restrict__ keys_in,
    const int32_t* __restrict__ vals_in, const int32_t* __restrict__ rb_in, int32_t n, int shift,
    const int32_t* __restrict__ offsets, int64_t ntiles, uint32_t* __restrict__ keys_out,
    int32_t* __restrict__ vals_out, int32_t* __restrict__ rb_out, const int32_t* counts) {
  if (counts[kErrFlags]) return;
  __shared__ int32_t running[kBins];
  __shared__ int32_t wcnt[kThreads / 64][kBins];
  const int t = threadIdx.x, w = t >> 6;
  const int64_t tile = xcd_tile(ntiles);
  if (tile < 0) return;
  running[t] = offsets[(int64_t)t * ntiles + tile];
#pragma unroll
  for (int k = 0; k < kThreads / 64; ++k) wcnt[k][t] = 0;
  __syncthreads();
  const uint64_t lt = lanemask_lt();
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = tile * kTile + j * kThreads + t;
    const bool valid = i < n;
    uint32_t key = 0;
    int32_t val = 0, rb = 0;
    int dg = 0;
    if (valid) {
      key = FIRST ? (0x7fffffffu - (uint32_t)d_in[i]) : keys_in[i];
      val = FIRST ? (int32_t)i : vals_in[i];
      rb = rb_in[i];
      dg = (key >> shift) & (kBins - 1);
    }
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (dg >> b) & 1;
      uint64_t bal = __ballot(valid && bit);
      m &= bit ? bal : ~bal;
    }
    const int rank = __popcll(m & lt);
    if (valid && rank == 0) wcnt[w][dg] = __popcll(m);
    __syncthreads();
    if (valid) {
      int32_t pos = running[dg] + rank;
      for (int k = 0; k < w; ++k) pos += wcnt[k][dg];
      if (pos >= 0 && pos < n) {
        keys_out[pos] = key;
        vals_out[pos] = val;
        rb_out[pos] = rb;
      } else {
        atomicOr(const_cast<int32_t*>(counts) + kErrFlags, kErrInternal);
      }
    }
    __syncthreads();
    int32_t tot = 0;
#pragma unroll
    for (int k = 0; k < kThreads / 64; ++k) {
      tot += wcnt[k][t];
      wcnt[k][t] = 0;
    }
    running[t] += tot;
    __syncthreads();
  }
}

template <class F>
__global__ __launch_bounds__(kThreads) void k_scan_reduce(F f, int64_t n_host,
                                                          const int32_t* n_dev,
                                                          int32_t* tile_sums,
                                                          const int32_t* counts) {
  if (counts[kErrFlags]) return;
  const int64_t n = n_dev ? ((int64_t)*n_dev < n_host ? (int64_t)*n_dev : n_host) : n_host;
  const int64_t base = blockIdx.x * (int64_t)kTile + threadIdx.x * kItems;
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < kItems; ++k)
    if (base + k < n) s += f(base + k);
  int32_t tot;
  block_excl_scan<kThreads>(s, &tot);
  if (threadIdx.x == 0) tile_sums[blockIdx.x] = tot;
}

// exclusive scan of the tile sums by one workgroup of 1024 threads
__global__ __launch_bounds__(1024) void k_scan_tilesums(int32_t* ts, int64_t nt, int32_t* total,
                                                        const int32_t* counts) {
  if (counts[kErrFlags]) return;
  __shared__ int32_t carry_s;
  if (threadIdx.x == 0) carry_s = 0;
  __syncthreads();
  for (int64_t base = 0; base < nt; base += 1024) {
    const int64_t i = base + threadIdx.x;
    const int32_t v = i < nt ? ts[i] : 0;
    int32_t tot;
    const int32_t ex = block_excl_scan<1024>(v, &tot);
    const int32_t carry = carry_s;
    if (i < nt) ts[i] = carry + ex;
    __syncthreads();
    if (threadIdx.x == 0) carry_s = carry + tot;
    __syncthreads();
  }
  if (threadIdx.x == 0 && total) *total = carry_s;
}

template <class F>
__global__ __launch_bounds__(kThreads) void k_scan_apply(F f, int64_t n_host,
                                                         const int32_t* n_dev,
                                                         const int32_t* tile_sums,
                                                         int32_t* out, const int32_t* counts) {
  if (counts[kErrFlags]) return;
  const int64_t n = n_dev ? ((int64_t)*n_dev < n_host ? (int64_t)*n_dev : n_host) : n_host;
  const int64_t base = blockIdx.x * (int64_t)kTile + threadIdx.x * kItems;
  int32_t v[kItems];
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < kItems; ++k) {
    v[k] = base + k < n ? f(base + k) : 0;
    s += v[k];
  }
  int32_t tot;
  int32_t run = block_excl_scan<kThreads>(s, &tot) + tile_sums[blockIdx.x];
#pragma unroll
  for (int k = 0; k < kItems; ++k) {
    if (base + k < n) out[base + k] = run;
    run += v[k];
  }
}

__global__ __launch_bounds__(kThreads) void k_segments(const uint32_t* __restrict__ keys,
                                                       const int32_t* __restrict__ rbeg,
                                                       const int32_t* __restrict__ perm,
                                                       const int32_t* __restrict__ first,
                                                       int32_t V, int32_t T, int64_t max_seg,
                                                       int32_t* seg_row, int32_t* seg_beg,
                                                       int32_t* seg_end, int32_t* counts) {
  if (counts[kErrFlags]) return;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < V;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = perm[i];
    if (v < 0 || v >= V) {
      atomicOr(&counts[kErrFlags], kErrInternal);
      return;
    }
    const int32_t d = key_degree(keys[i]);
    const int32_t f = first[i];
    const int32_t ns = d > T ? (d + T - 1) / T : 1;
    if (f < 0 || (int64_t)f + ns > max_seg) {
      atomicOr(&counts[kErrFlags], kErrInternal);
      return;
    }
    const int32_t b0 = rbeg[i], e0 = b0 + d;
    for (int32_t j = 0; j < ns; ++j) {
      const int32_t b = b0 + j * T;
      seg_row[f + j] = v;
      seg_beg[f + j] = b;
      seg_end[f + j] = (e0 - b) > T ? b + T : e0;
    }
    const bool split = d > T;
    const bool next_split = (i + 1 < V) && key_degree(keys[i + 1]) > T;
    if (split && !next_split) {
      counts[kNSplit] = (int32_t)(i + 1);
      counts[kSSplit] = f + ns;
    }
    if (i == V - 1) counts[kNumSegments] = f + ns;
  }
}

// block b holds the segments s with floor(P(s) / B) == b; consecutive
// segments differ in P by at most seg_len + row_cost <= B, so no block id
// is skipped.
__global__ __launch_bounds__(kThreads) void k_blocks(const int32_t* __restrict__ P, int32_t B,
                                                     int64_t max_seg, int64_t max_blocks,
                                                     int32_t* block_ptr, int32_t* counts) {
  if (counts[kErrFlags]) return;
  const int32_t S = counts[kNumSegments];
  if (S > max_seg) {
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&counts[kErrFlags], kErrInternal);
    return;
  }
  for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < S;
       s += (int64_t)gridDim.x * blockDim.x) {
    const int32_t b = P[s] / B;
    if (b < 0 || b >= max_blocks) {
      atomicOr(&counts[kErrFlags], kErrInternal);
      return;
    }
    if (s == 0 || P[s - 1] / B != b) block_ptr[b] = (int32_t)s;
    if (s == S - 1) {
      block_ptr[b + 1] = S;
      counts[kNumBlocks] = b + 1;
    }
  }
}

template <class F>
void scan(F f, int64_t n_host, const int32_t* n_dev, int32_t* out, int32_t* total,
          int32_t* tile_sums, const int32_t* counts, hipStream_t st) {
  const int64_t nt = cdiv(n_host, kTile);
  if (nt == 0) return;
  hipLaunchKernelGGL(k_scan_reduce<F>, dim3(nt), dim3(kThreads), 0, st, f, n_host, n_dev,
                     tile_sums, counts);
  hipLaunchKernelGGL(k_scan_tilesums, dim3(1), dim3(1024), 0, st, tile_sums, nt, total, counts);
  hipLaunchKernelGGL(k_scan_apply<F>, dim3(nt), dim3(kThreads), 0, st, f, n_host, n_dev,
                     tile_sums, out, counts);
}

inline unsigned grid_for(int64_t n, int64_t cap = 16384) {
  int64_t g = cdiv(n, kThreads);
  if (g < 1) g = 1;
  return (unsigned)(g < cap ? g : cap);
}

}  // namespace

bool plan_layout(int32_t V, int32_t Vs, int64_t E, int32_t T, int32_t B, int32_t c,
                 PlanLayout* L) {
  if (V < 0 || Vs < 0 || E < 0 || E >= (int64_t(1) << 31) || T <= 0 || c <= 0 || B < T + c)
    return false;
  L->max_segments = (int64_t)V + cdiv(E, T);
  const int64_t ptot = E + (int64_t)c * L->max_segments;
  if (ptot >= (int64_t(1) << 31) - 1) return false;
  L->max_blocks = ptot / B + 1;
  L->max_split = E / (int64_t(T) + 1) < V ? E / (int64_t(T) + 1) : V;
  L->max_split_segments = cdiv(E, T) + L->max_split;
  L->radix_tiles = cdiv(V, kTile);
  L->scan_tiles_rows = cdiv(V, kTile);
  L->scan_tiles_segs = cdiv(L->max_segments, kTile);
  const int64_t hist_n = (int64_t)kBins * L->radix_tiles;
  L->outdeg_nb = cdiv(Vs, kBucketSize);
  L->edge_tiles = cdiv(E, kEdgeTile);
  L->outdeg_bucketed = L->outdeg_nb <= kMaxBuckets && E > 0;
  int64_t scan_tiles = cdiv(hist_n, kTile);
  if (L->outdeg_bucketed && cdiv(L->outdeg_nb * L->edge_tiles, kTile) > scan_tiles)
    scan_tiles = cdiv(L->outdeg_nb * L->edge_tiles, kTile);
  if (L->scan_tiles_rows > scan_tiles) scan_tiles = L->scan_tiles_rows;
  if (L->scan_tiles_segs > scan_tiles) scan_tiles = L->scan_tiles_segs;

  size_t o = 0;
  auto take = [&](int64_t n_int) {
    size_t at = o;
    o = align256(o + (size_t)n_int * 4);
    return at;
  };
  L->off_d_in = take(V);
  L->off_d_out = take(Vs);
  L->off_perm = take(V);
  L->off_first = take((int64_t)V + 1);
  L->off_seg_row = take(L->max_segments);
  L->off_seg_beg = take(L->max_segments);
  L->off_seg_end = take(L->max_segments);
  L->off_block_ptr = take(L->max_blocks + 1);
  L->off_counts = take(kCountSlots);
  L->off_scratch = o;
  // scratch: keysA, valsA, keysB, valsB, row begins A and B, hist, tile
  // sums, cost prefix, bucketed source ids, bucket histogram
  take(V); take(V); take(V); take(V); take(V); take(V);
  take(hist_n);
  take(scan_tiles + 1);
  take(L->outdeg_bucketed ? scan_tiles + 1 : 0);  // tile sums of the out-degree branch
  take(L->max_segments);
  take(L->outdeg_bucketed ? cdiv(E, 2) : 0);
  take(L->outdeg_bucketed ? L->outdeg_nb * L->edge_tiles : 0);
  take(L->outdeg_bucketed ? (int64_t)kOutdegSplit * L->outdeg_nb * kBucketSize : 0);
  L->scratch_bytes = o - L->off_scratch;
  L->total = o;
  return true;
}

hipError_t launch_plan_build(const saga_plan& p, const PlanLayout& L, hipStream_t st,
                             hipStream_t order_st, hipEvent_t fork, hipEvent_t join) {
  const int32_t V = p.num_dst, Vs = p.num_src, T = p.seg_len;
  const int64_t E = p.num_edges;
  char* sc = static_cast<char*>(p.scratch);
  size_t o = 0;
  auto take = [&](int64_t n_int) {
    char* at = sc + o;
    o = align256(o + (size_t)n_int * 4);
    return at;
  };
  uint32_t* keysA = reinterpret_cast<uint32_t*>(take(V));
  int32_t* valsA = reinterpret_cast<int32_t*>(take(V));
  uint32_t* keysB = reinterpret_cast<uint32_t*>(take(V));
  int32_t* valsB = reinterpret_cast<int32_t*>(take(V));
  int32_t* rbA = reinterpret_cast<int32_t*>(take(V));
  int32_t* rbB = reinterpret_cast<int32_t*>(take(V));
  const int64_t ntiles = L.radix_tiles;
  int32_t* hist = reinterpret_cast<int32_t*>(take((int64_t)kBins * ntiles));
  int64_t scan_tiles = cdiv((int64_t)kBins * ntiles, kTile);
  if (L.scan_tiles_rows > scan_tiles) scan_tiles = L.scan_tiles_rows;
  if (L.scan_tiles_segs > scan_tiles) scan_tiles = L.scan_tiles_segs;
  if (L.outdeg_bucketed && cdiv(L.outdeg_nb * L.edge_tiles, kTile) > scan_tiles)
    scan_tiles = cdiv(L.outdeg_nb * L.edge_tiles, kTile);
  int32_t* tile_sums = reinterpret_cast<int32_t*>(take(scan_tiles + 1));
  int32_t* tile_sums2 = reinterpret_cast<int32_t*>(take(L.outdeg_bucketed ? scan_tiles + 1 : 0));
  int32_t* P = reinterpret_cast<int32_t*>(take(L.max_segments));
  uint16_t* bucketed = reinterpret_cast<uint16_t*>(take(L.outdeg_bucketed ? cdiv(E, 2) : 0));
  int32_t* ohist = reinterpret_cast<int32_t*>(take(L.outdeg_bucketed ? L.outdeg_nb * L.edge_tiles : 0));
  int32_t* opart = reinterpret_cast<int32_t*>(
      take(L.outdeg_bucketed ? (int64_t)kOutdegSplit * L.outdeg_nb * kBucketSize : 0));

  hipLaunchKernelGGL(k_zero, dim3(1), dim3(64), 0, st, p.counts, (int64_t)kCountSlots);
  if (Vs > 0 && !L.outdeg_bucketed)
    hipLaunchKernelGGL(k_zero, dim3(grid_for(Vs)), dim3(kThreads), 0, st, p.d_out, (int64_t)Vs);
  // Two independent branches: the out-degree count (col_idx only) and the
  // row order (row_ptr only: in-degrees, CSR validation, degree sort,
  // segments, row blocks).  With an order stream, the row order runs there
  // after the counters are cleared, so that whatever the caller enqueues on
  // `st` after the out-degrees (the d_out-scaled transform) overlaps it.
  // The graphs whose out-degrees are counted inside k_degrees (no buckets)
  // run both on `st`.
  const bool split = order_st && fork && join && L.outdeg_bucketed && V > 0;
  hipStream_t qst = st;
  if (split) {
    hipError_t e = hipEventRecord(fork, st);
    if (e == hipSuccess) e = hipStreamWaitEvent(order_st, fork, 0);
    if (e != hipSuccess) return e;
    qst = order_st;
  }
  if (V == 0) {
    if (join) {
      hipError_t e = hipEventRecord(join, st);
      if (e != hipSuccess) return e;
    }
    return hipGetLastError();
  }
  const int edges_too = L.outdeg_bucketed ? 0 : 1;
  hipLaunchKernelGGL(k_degrees, dim3(grid_for(edges_too && E > V ? E : V, 2048)), dim3(kThreads), 0, qst,
                     p.row_ptr, p.col_idx, V, Vs, E, edges_too, p.d_in, p.d_out, p.counts);
  if (L.outdeg_bucketed) {
    const int nb = (int)L.outdeg_nb;
    const int64_t et = L.edge_tiles;
    hipLaunchKernelGGL(k_outdeg_hist, dim3(xcd_grid(et)), dim3(kThreads), (kThreads / 64) * nb * 4, st,
                       p.col_idx, E, Vs, nb, ohist, et, p.counts);
    scan(ArrF{ohist}, (int64_t)nb * et, nullptr, ohist, nullptr, tile_sums2, p.counts, st);
    hipLaunchKernelGGL(k_outdeg_scatter, dim3(xcd_grid(et)), dim3(kThreads),
                       3 * nb * 4 + 2 * kEdgeTile * 2, st, p.col_idx, E, nb, ohist, et, bucketed,
                       p.counts);
    hipLaunchKernelGGL(k_outdeg_count, dim3(kOutdegSplit, nb), dim3(1024), 0, st, bucketed, ohist,
                       et, nb, E, Vs, opart, p.counts);
    hipLaunchKernelGGL(k_outdeg_reduce, dim3(grid_for(Vs)), dim3(kThreads), 0, st, opart, nb, Vs,
                       p.d_out, p.counts);
  }
  st = qst;  // the row order

  // degree order: 4 stable passes of 8 bits over key = 0x7fffffff - d_in;
  // the sorted keys end in keysB, the row begins in rbB
  const uint32_t* kin[4] = {nullptr, keysA, keysB, keysA};
  const int32_t* vin[4] = {nullptr, valsA, valsB, valsA};
  const int32_t* rin[4] = {p.row_ptr, rbA, rbB, rbA};
  uint32_t* kout[4] = {keysA, keysB, keysA, keysB};
  int32_t* vout[4] = {valsA, valsB, valsA, p.perm};
  int32_t* rout[4] = {rbA, rbB, rbA, rbB};
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 8 * pass;
    if (pass == 0)
      hipLaunchKernelGGL(k_radix_hist<true>, dim3(xcd_grid(ntiles)), dim3(kThreads), 0, st, p.d_in,
                         kin[pass], V, shift, hist, ntiles, p.counts);
    else
      hipLaunchKernelGGL(k_radix_hist<false>, dim3(xcd_grid(ntiles)), dim3(kThreads), 0, st, p.d_in,
                         kin[pass], V, shift, hist, ntiles, p.counts);
    scan(ArrF{hist}, (int64_t)kBins * ntiles, nullptr, hist, nullptr, tile_sums, p.counts, st);
    if (pass == 0)
      hipLaunchKernelGGL((k_radix_scatter<true>), dim3(xcd_grid(ntiles)), dim3(kThreads), 0, st,
                         p.d_in, kin[pass], vin[pass], rin[pass], V, shift, hist, ntiles,
                         kout[pass], vout[pass], rout[pass], p.counts);
    else
      hipLaunchKernelGGL((k_radix_scatter<false>), dim3(xcd_grid(ntiles)), dim3(kThreads), 0, st,
                         p.d_in, kin[pass], vin[pass], rin[pass], V, shift, hist, ntiles,
                         kout[pass], vout[pass], rout[pass], p.counts);
  }

  // segments per row in perm order -> row_seg_first (total at [V])
  scan(NsegF{keysB, T}, V, nullptr, p.row_seg_first, p.row_seg_first + V, tile_sums, p.counts, st);
  hipLaunchKernelGGL(k_segments, dim3(grid_for(V)), dim3(kThreads), 0, st, keysB, rbB, p.perm,
                     p.row_seg_first, V, T, L.max_segments, p.seg_row, p.seg_beg, p.seg_end,
                     p.counts);
  // cost prefix over segments -> row blocks
  scan(CostF{p.seg_beg, p.seg_end, p.row_cost}, L.max_segments, p.counts + kNumSegments, P,
       nullptr, tile_sums, p.counts, st);
  hipLaunchKernelGGL(k_blocks, dim3(grid_for(L.max_segments)), dim3(kThreads), 0, st, P,
                     p.block_cost, L.max_segments, L.max_blocks, p.block_ptr, p.counts);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && join) e = hipEventRecord(join, st);
  return e;
}

}  // namespace saga
