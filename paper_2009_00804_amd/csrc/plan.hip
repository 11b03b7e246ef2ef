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
// instead: (1) each tile of kOdTile CSR entries is sorted by bucket (the
// source id's high bits, kOdBucket ids per bucket) in LDS and written back
// to its own place in one contiguous piece, as 16-bit offsets within the
// bucket, with the start of every bucket's run in the tile; (2) per bucket,
// workgroups count their share of the tiles' runs into an LDS histogram and
// store it; (3) the partial histograms are summed.  Counting is order-free,
// so no global scan is needed and every global write is contiguous.
// ------------------------------------------------------------------------
// Tile of this workgroup in an XCD-blocked order.  Workgroups are handed to
// the eight XCDs in turn (w % 8), so with tile = w the tiles one L2 sees are
// eight apart, and the tile-minor entries of neighbouring tiles (32 to a
// 128-byte line) are written and read as partial lines through eight
// different L2s.  Here XCD x takes the contiguous run [x * per, (x + 1) *
// per) of tiles.  The grid is xcd_grid(ntiles) workgroups; the spare ones
// get -1.  Any dispatch order gives the same result; only the locality
// depends on it.
constexpr int kXcds = 8;
__device__ __forceinline__ int64_t xcd_tile(int64_t ntiles) {
  const int64_t per = (ntiles + kXcds - 1) / kXcds;
  const int64_t w = blockIdx.x, t = (w % kXcds) * per + w / kXcds;
  return t < ntiles ? t : -1;
}
inline unsigned xcd_grid(int64_t ntiles) {
  return (unsigned)(kXcds * ((ntiles + kXcds - 1) / kXcds));
}

// Shapes measured on the 2^21-source R-MAT graph (E = 1.07e8), whole
// out-degree count: 16,384 ids per bucket and tiles of 16,384 entries; the
// count with about 1024 workgroups (two per CU, 64 KB of LDS each), each
// wave reading 4 tiles' runs at a time, 256 entries of each before counting.
// 8,192 or 32,768 ids per bucket, 256 or 512 count workgroups, 8 x 2 or
// 16 x 1 runs x loads, 32-bit loads of entry pairs, and persistent bin
// workgroups that prefetch their next tile were all slower.
constexpr int kOdBits = 14;
constexpr int kOdBucket = 1 << kOdBits;
constexpr int64_t kOdMaxSources = int64_t(1) << 23;  // larger graphs count in k_degrees
constexpr int kOdMaxBuckets = (int)(kOdMaxSources >> kOdBits);
constexpr int kOdThreads = 512, kOdWaves = kOdThreads / 64;
constexpr int kOdItems = 32;
constexpr int kOdTile = kOdThreads * kOdItems;  // 16384 entries per tile
constexpr int kOdCountWgs = 1024, kOdRuns = 4, kOdLoads = 4;
static_assert(kOdBits <= 15, "the count's LDS histogram holds 2^15 counters");
static_assert(kOdTile <= 65536, "16-bit offsets");
static_assert(64 * kOdItems < 0xffff, "16-bit ranks within a wave");
// workgroups per bucket in the count: about kOdCountWgs workgroups in all
inline int outdeg_split(int64_t nb) {
  const int64_t s = nb >= kOdCountWgs || nb < 1 ? 1 : kOdCountWgs / nb;
  return (int)(s > 16 ? 16 : s);
}
inline size_t outdeg_bin_lds(int nb) {
  return (size_t)kOdWaves * nb * 4 + (size_t)kOdTile * 2;
}
static_assert((size_t)kOdWaves * kOdMaxBuckets * 4 + (size_t)kOdTile * 2 + 64 <= 65536,
              "the bin kernel's LDS stays within 64 KB");

// Sort one tile by bucket.  Each wave ranks its own entries with counters
// of its own, laid out wave-major (a wave's lanes hit nb consecutive words);
// the bucket-major scan over (bucket, wave) then places bucket b's entries of
// wave 0, 1, ... one after another.  loc[b * ntiles + tile] is the start of
// bucket b's run within the tile, loc[nb * ntiles + tile] the tile's valid
// entries.  Source ids outside [0, Vs) raise error bit 8 and are left out.
// The loads are unconditional (E > 0, so a tile holds at least one entry):
// an entry past the tile's end reads the tile's last one and is then
// ignored, so no branch splits the batch of loads.
__global__ __launch_bounds__(kOdThreads) void k_outdeg_bin(const int32_t* __restrict__ col,
                                                           int64_t E, int32_t Vs, int nb,
                                                           int64_t ntiles,
                                                           uint16_t* __restrict__ out,
                                                           int32_t* __restrict__ loc,
                                                           int32_t* counts) {
  extern __shared__ int32_t sm[];
  int32_t* cnt = sm;  // [kOdWaves][nb]
  uint16_t* sval = reinterpret_cast<uint16_t*>(sm + kOdWaves * nb);  // [kOdTile]
  __shared__ int32_t wsum[kOdWaves];
  const int64_t tile = xcd_tile(ntiles);
  if (tile < 0) return;
  const int tx = threadIdx.x, wave = tx >> 6, lane = tx & 63;
  const int64_t base = tile * (int64_t)kOdTile;
  const int n = E - base < kOdTile ? (int)(E - base) : kOdTile;
  for (int b = tx; b < kOdWaves * nb; b += kOdThreads) cnt[b] = 0;
  const int32_t* p = col + base;
  int32_t c[kOdItems];
  if (n == kOdTile) {
#pragma unroll
    for (int j = 0; j < kOdItems; ++j) c[j] = __builtin_nontemporal_load(p + j * kOdThreads + tx);
  } else {
#pragma unroll
    for (int j = 0; j < kOdItems; ++j) {
      const int i = j * kOdThreads + tx;
      c[j] = __builtin_nontemporal_load(p + (i < n ? i : n - 1));
    }
  }
  __syncthreads();
  // rank within (wave, bucket), two 16-bit ranks to a register (a wave
  // ranks at most 64 * kOdItems entries); 0xffff marks no entry
  int32_t* cw = cnt + wave * nb;
  uint32_t r[kOdItems / 2];
  int err = 0;
#pragma unroll
  for (int j = 0; j < kOdItems; ++j) {
    const bool in = j * kOdThreads + tx < n;
    const bool ok = in && c[j] >= 0 && c[j] < Vs;
    err |= in && !ok;
    const uint32_t rj = ok ? (uint32_t)atomicAdd(&cw[c[j] >> kOdBits], 1) : 0xffffu;
    r[j / 2] = j % 2 ? r[j / 2] | rj << 16 : rj;
  }
  if (__any(err) && lane == 0) atomicOr(&counts[kErrFlags], 8);
  __syncthreads();
  {  // exclusive scan over k = b * kOdWaves + w (entry cnt[w * nb + b]):
     // thread t owns k in [t * pk, (t + 1) * pk), then a wave scan and a
     // cross-wave pass
    const int m = kOdWaves * nb;
    const int pk = (m + kOdThreads - 1) / kOdThreads;
    const int k0 = tx * pk;
    int32_t own = 0;
    for (int k = k0; k < k0 + pk && k < m; ++k) own += cnt[(k % kOdWaves) * nb + k / kOdWaves];
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
    for (int k = k0; k < k0 + pk && k < m; ++k) {
      const int a = (k % kOdWaves) * nb + k / kOdWaves;
      const int32_t v = cnt[a];
      cnt[a] = run;
      if (k % kOdWaves == 0) loc[(int64_t)(k / kOdWaves) * ntiles + tile] = run;
      run += v;
    }
    if (tx == kOdThreads - 1) loc[(int64_t)nb * ntiles + tile] = run;
  }
  __syncthreads();
  int32_t total = 0;
  for (int w = 0; w < kOdWaves; ++w) total += wsum[w];
#pragma unroll
  for (int j = 0; j < kOdItems; ++j) {
    const uint32_t rj = r[j / 2] >> (16 * (j % 2)) & 0xffffu;
    if (rj != 0xffffu) sval[cw[c[j] >> kOdBits] + (int)rj] = (uint16_t)(c[j] & (kOdBucket - 1));
  }
  __syncthreads();
  // the tile's sorted entries, 8 to a 16-byte store
  const int nv = total >> 3;
  uint4* out4 = reinterpret_cast<uint4*>(out + base);
  const uint4* s4 = reinterpret_cast<const uint4*>(sval);
  for (int i = tx; i < nv; i += kOdThreads) out4[i] = s4[i];
  for (int i = nv * 8 + tx; i < total; i += kOdThreads) out[base + i] = sval[i];
}

// Bucket b's entries, from the runs of tiles [t0, t1) (slice s of
// outdeg_split(nb)), counted into LDS; the histogram goes to
// part[s][b * kOdBucket + i].  Each wave takes R tiles at a time and reads
// the first J * 64 entries of each run before counting, so that R * J loads
// are in flight; longer runs finish in a loop.
__global__ __launch_bounds__(1024) void k_outdeg_count(const uint16_t* __restrict__ bk,
                                                       const int32_t* __restrict__ loc,
                                                       int64_t ntiles, int nb, int64_t E,
                                                       int32_t* __restrict__ part,
                                                       const int32_t* counts) {
  if (counts[kErrFlags]) return;
  __shared__ int32_t h[kOdBucket];
  constexpr int R = kOdRuns, J = kOdLoads, NW = 1024 / 64;
  // buckets in an XCD-blocked order (gridDim.x = xcd_grid(nb)): XCD x takes
  // the contiguous buckets [x * per, (x + 1) * per), so that neighbouring
  // buckets, whose runs share the 128-byte lines where they meet, read them
  // through one L2
  const int per = (int)((nb + kXcds - 1) / kXcds);
  const int b = (int)(blockIdx.x % kXcds) * per + (int)(blockIdx.x / kXcds);
  const int s = blockIdx.y, S = gridDim.y;
  if (b >= nb) return;
  for (int i = threadIdx.x; i < kOdBucket; i += 1024) h[i] = 0;
  __syncthreads();
  const int64_t t0 = ntiles * s / S, t1 = ntiles * (s + 1) / S;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int32_t* lb = loc + (int64_t)b * ntiles;
  const int32_t* le = loc + (int64_t)(b + 1) * ntiles;
  for (int64_t tg = t0 + (int64_t)wave * R; tg < t1; tg += (int64_t)NW * R) {
    int64_t beg[R];
    int32_t len[R];
#pragma unroll
    for (int q = 0; q < R; ++q) {
      const int64_t t = tg + q;
      len[q] = 0;
      beg[q] = 0;
      if (t < t1) {
        const int64_t tbase = t * (int64_t)kOdTile;
        const int32_t n = (int32_t)(E - tbase < kOdTile ? E - tbase : kOdTile);
        int32_t lo = lb[t], hi = le[t];
        lo = lo < 0 ? 0 : (lo > n ? n : lo);
        hi = hi < lo ? lo : (hi > n ? n : hi);
        beg[q] = tbase + lo;
        len[q] = hi - lo;
      }
    }
    uint32_t v[R][J];
#pragma unroll
    for (int q = 0; q < R; ++q)
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int k = j * 64 + lane;
        v[q][j] = k < len[q] ? (uint32_t)bk[beg[q] + k] : 0xffffffffu;
      }
#pragma unroll
    for (int q = 0; q < R; ++q)
#pragma unroll
      for (int j = 0; j < J; ++j)
        if (v[q][j] != 0xffffffffu) atomicAdd(&h[v[q][j] & (kOdBucket - 1)], 1);
#pragma unroll
    for (int q = 0; q < R; ++q)
      for (int k = J * 64 + lane; k < len[q]; k += 64)
        atomicAdd(&h[bk[beg[q] + k] & (kOdBucket - 1)], 1);
  }
  __syncthreads();
  int32_t* pw = part + (int64_t)s * nb * kOdBucket + (int64_t)b * kOdBucket;
  for (int i = threadIdx.x; i < kOdBucket; i += 1024) pw[i] = h[i];
}

// d_out[v] = the sum of the S partial counts, four sources per thread as
// 16-byte loads (part and d_out are 256-byte aligned, stride a multiple of 4)
__global__ __launch_bounds__(kThreads) void k_outdeg_reduce(const int32_t* __restrict__ part,
                                                            int nb, int S, int32_t Vs,
                                                            int32_t* __restrict__ d_out,
                                                            const int32_t* counts) {
  if (counts[kErrFlags]) return;
  const int64_t stride = (int64_t)nb * kOdBucket;
  const int64_t n4 = Vs / 4;
  const int64_t g0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x, gs = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = g0; i < n4; i += gs) {
    int4 sum = make_int4(0, 0, 0, 0);
    for (int w = 0; w < S; ++w) {
      const int4 x = reinterpret_cast<const int4*>(part + w * stride)[i];
      sum.x += x.x;
      sum.y += x.y;
      sum.z += x.z;
      sum.w += x.w;
    }
    reinterpret_cast<int4*>(d_out)[i] = sum;
  }
  for (int64_t v = 4 * n4 + g0; v < Vs; v += gs) {
    int32_t sum = 0;
    for (int w = 0; w < S; ++w) sum += part[w * stride + v];
    d_out[v] = sum;
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
  L->outdeg_nb = cdiv(Vs, kOdBucket);
  L->edge_tiles = cdiv(E, kOdTile);
  L->outdeg_bucketed = L->outdeg_nb > 0 && L->outdeg_nb <= kOdMaxBuckets && E > 0;
  int64_t scan_tiles = cdiv(hist_n, kTile);
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
  // sums, cost prefix, bucketed source ids, bucket run starts, partial
  // out-degree histograms
  const bool bk = L->outdeg_bucketed;
  take(V); take(V); take(V); take(V); take(V); take(V);
  take(hist_n);
  take(scan_tiles + 1);
  take(L->max_segments);
  take(bk ? cdiv(E, 2) : 0);
  take(bk ? (L->outdeg_nb + 1) * L->edge_tiles : 0);
  take(bk ? (int64_t)outdeg_split(L->outdeg_nb) * L->outdeg_nb * kOdBucket : 0);
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
  int32_t* tile_sums = reinterpret_cast<int32_t*>(take(scan_tiles + 1));
  int32_t* P = reinterpret_cast<int32_t*>(take(L.max_segments));
  const bool bk = L.outdeg_bucketed;
  uint16_t* bucketed = reinterpret_cast<uint16_t*>(take(bk ? cdiv(E, 2) : 0));
  int32_t* oloc = reinterpret_cast<int32_t*>(take(bk ? (L.outdeg_nb + 1) * L.edge_tiles : 0));
  int32_t* opart = reinterpret_cast<int32_t*>(
      take(bk ? (int64_t)outdeg_split(L.outdeg_nb) * L.outdeg_nb * kOdBucket : 0));

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
    const int S = outdeg_split(nb);
    hipLaunchKernelGGL(k_outdeg_bin, dim3(xcd_grid(et)), dim3(kOdThreads), outdeg_bin_lds(nb), st,
                       p.col_idx, E, Vs, nb, et, bucketed, oloc, p.counts);
    hipLaunchKernelGGL(k_outdeg_count, dim3(xcd_grid(nb), S), dim3(1024), 0, st, bucketed, oloc, et,
                       nb, E, opart, p.counts);
    hipLaunchKernelGGL(k_outdeg_reduce, dim3(grid_for((Vs + 3) / 4)), dim3(kThreads), 0, st, opart, nb,
                       S, Vs, p.d_out, p.counts);
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
