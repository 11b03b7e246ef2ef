// Typed-edge layout of R-GCN (Table I, R-GCN row: Scatter takes the edge and
// its source, ApplyEdge is an MLP chosen by the edge's type; Sec. 3.2
// "ApplyEdge": the edges of one type are selected and batched into one
// GEMM).
//
// The per-edge transform x_u W_r depends only on the (relation r, source u)
// pair, so it is computed once per distinct pair that some edge carries, as
// one grouped matrix-core GEMM over all relations (gemm.hip).  This file
// builds, on the device, what that GEMM and the typed Gather need:
//   rel_count[r]   distinct sources of relation r
//   rel_ptr[r]     first pair row of relation r; ranges padded to whole
//                  GEMM tiles (kRelTile rows), so that a tile never mixes
//                  two relations' weights
//   pair_src[q]    source vertex of pair row q (-1 in the padding)
//   edge_pair[e]   pair row of CSR entry e
//   edge_norm[e]   1 / c(v, r): c counts the in-edges of v with e's type
//
// Pairs are found without sorting: one bit per (relation, source) in a
// bitmap (relation-major, each relation's words padded to whole counting
// blocks), set by the edges -- through byte flags packed into bits when the
// flags fit in 256 MB, else by bitmap atomics.  The pair row of a set bit is
// the number of set bits before it in its relation plus the relation's
// offset: a scan of block popcounts, then of word popcounts, then a popcount
// under a mask.  The per-row type counts use LDS histograms (one per
// workgroup for the long rows, one per wave for the others).
#include <algorithm>

#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kThreads = 256;
constexpr int kBlockWords = 1024;  // bitmap words per counting block (4 per thread)

__device__ __forceinline__ void lds_wait() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
  asm volatile("" ::: "memory");
}

__global__ void k_rel_fill(uint32_t* __restrict__ p, int64_t n, uint32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// one bit per (relation, source) pair carried by some edge; out-of-range
// types raise the error flag and set nothing
__global__ __launch_bounds__(kThreads) void k_rel_mark(const int32_t* __restrict__ col,
                                                       const int32_t* __restrict__ et, int64_t E,
                                                       int R, int64_t wp, uint32_t* bm,
                                                       const int32_t* __restrict__ plan_counts,
                                                       int32_t* rcounts) {
  if (plan_counts[kErrFlags]) return;
  bool bad = false;
  for (int64_t e = blockIdx.x * (int64_t)kThreads + threadIdx.x; e < E;
       e += (int64_t)gridDim.x * kThreads) {
    const int r = et[e];
    if (r < 0 || r >= R) {
      bad = true;
      continue;
    }
    const int u = col[e];
    uint32_t* w = bm + (int64_t)r * wp + (u >> 5);
    const uint32_t bit = 1u << (u & 31);
    // most edges of a hub source find their bit already set: read first
    if (!(__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & bit))
      atomicOr(w, bit);
  }
  if (bad) atomicOr(&rcounts[kRelErr], 1);
}

// set bits of each counting block
__global__ __launch_bounds__(kThreads) void k_rel_bcount(const uint32_t* __restrict__ bm,
                                                         int64_t nblocks, int32_t* __restrict__ bcnt,
                                                         const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  __shared__ int red[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const uint4 v = reinterpret_cast<const uint4*>(bm + b * kBlockWords)[threadIdx.x];
    int c = __popc(v.x) + __popc(v.y) + __popc(v.z) + __popc(v.w);
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
    if (lane == 0) red[wave] = c;
    __syncthreads();
    if (threadIdx.x == 0) bcnt[b] = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
  }
}

// One workgroup.  Thread t owns relations [t * rpt, (t + 1) * rpt): it sums
// their block counts (rel_count), the tile-padded sizes are scanned across
// threads (rel_ptr), and each relation's blocks get their first pair row.
__global__ __launch_bounds__(1024) void k_rel_scan(const int32_t* __restrict__ bcnt, int R,
                                                   int64_t bpr, int tile,
                                                   int32_t* __restrict__ rel_count,
                                                   int32_t* __restrict__ rel_ptr,
                                                   int32_t* __restrict__ block_base,
                                                   int32_t* __restrict__ rcounts,
                                                   const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  __shared__ int64_t s_pad[1024];
  __shared__ int64_t s_cnt[1024];
  const int t = threadIdx.x;
  const int rpt = (R + 1023) / 1024;
  int64_t pad = 0, cnt = 0;
  for (int k = 0; k < rpt; ++k) {
    const int r = t * rpt + k;
    if (r < R) {
      int64_t q = 0;
      for (int64_t j = 0; j < bpr; ++j) q += bcnt[(int64_t)r * bpr + j];
      rel_count[r] = (int32_t)q;
      pad += (q + tile - 1) / tile * tile;
      cnt += q;
    }
  }
  // inclusive scan of pad (and a running total of cnt) over the threads
  s_pad[t] = pad;
  s_cnt[t] = cnt;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int64_t a = t >= off ? s_pad[t - off] : 0;
    const int64_t b = t >= off ? s_cnt[t - off] : 0;
    __syncthreads();
    s_pad[t] += a;
    s_cnt[t] += b;
    __syncthreads();
  }
  int64_t base = s_pad[t] - pad;
  for (int k = 0; k < rpt; ++k) {
    const int r = t * rpt + k;
    if (r < R) {
      rel_ptr[r] = (int32_t)base;
      int64_t run = base;
      for (int64_t j = 0; j < bpr; ++j) {
        block_base[(int64_t)r * bpr + j] = (int32_t)run;
        run += bcnt[(int64_t)r * bpr + j];
      }
      const int64_t q = rel_count[r];
      base += (q + tile - 1) / tile * tile;
    }
  }
  if (t == 1023) {
    rel_ptr[R] = (int32_t)s_pad[1023];
    rcounts[kRelRows] = (int32_t)s_pad[1023];
    rcounts[kRelPairs] = (int32_t)s_cnt[1023];
  }
}

// pair row of every set bit: word_base[w] = pair row of the first set bit of
// word w; pair_src[row] = the source the bit stands for
__global__ __launch_bounds__(kThreads) void k_rel_pairs(const uint32_t* __restrict__ bm,
                                                        int64_t nblocks, int64_t wp,
                                                        const int32_t* __restrict__ block_base,
                                                        int32_t* __restrict__ word_base,
                                                        int32_t* __restrict__ pair_src,
                                                        const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  __shared__ int wsum[kThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const int64_t w0 = b * kBlockWords + threadIdx.x * 4;
    const uint4 v = *reinterpret_cast<const uint4*>(bm + w0);
    const uint32_t x[4] = {v.x, v.y, v.z, v.w};
    const int c = __popc(x[0]) + __popc(x[1]) + __popc(x[2]) + __popc(x[3]);
    int incl = c;
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off, 64);
      if (lane >= off) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int woff = 0;
    for (int i = 0; i < wave; ++i) woff += wsum[i];
    int base = block_base[b] + woff + incl - c;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t w = w0 + k;
      word_base[w] = base;
      const int64_t u0 = (w % wp) * 32;
      uint32_t m = x[k];
      while (m) {
        pair_src[base++] = (int32_t)(u0 + __builtin_ctz(m));
        m &= m - 1;
      }
    }
    __syncthreads();  // wsum is rewritten for the next block
  }
}

// the padding rows of each relation's range
__global__ void k_rel_pad(const int32_t* __restrict__ rel_ptr,
                          const int32_t* __restrict__ rel_count, int R,
                          int32_t* __restrict__ pair_src, const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  for (int r = blockIdx.x; r < R; r += gridDim.x) {
    const int64_t a = (int64_t)rel_ptr[r] + rel_count[r], b = rel_ptr[r + 1];
    for (int64_t q = a + threadIdx.x; q < b; q += blockDim.x) pair_src[q] = -1;
  }
}

// pair row of every edge: the set bits of its relation before its own
__global__ __launch_bounds__(kThreads) void k_rel_edges(const int32_t* __restrict__ col,
                                                        const int32_t* __restrict__ et, int64_t E,
                                                        int R, int64_t wp,
                                                        const uint32_t* __restrict__ bm,
                                                        const int32_t* __restrict__ word_base,
                                                        int32_t* __restrict__ edge_pair,
                                                        const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  for (int64_t e = blockIdx.x * (int64_t)kThreads + threadIdx.x; e < E;
       e += (int64_t)gridDim.x * kThreads) {
    const int r = et[e];
    if (r < 0 || r >= R) {
      edge_pair[e] = 0;
      continue;
    }
    const int u = col[e];
    const int64_t w = (int64_t)r * wp + (u >> 5);
    edge_pair[e] = word_base[w] + __popc(bm[w] & ((1u << (u & 31)) - 1u));
  }
}

// The three passes over a row's types, STEP threads apart, four loads in
// flight per thread: count (LDS atomics), read back into edge_norm, clear.
template <int STEP>
__device__ __forceinline__ void count_types(const int32_t* __restrict__ et, int beg, int end, int t,
                                            int R, int32_t* hist) {
  for (int e0 = beg + t; e0 < end; e0 += 4 * STEP) {
    int r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = e0 + j * STEP < end ? et[e0 + j * STEP] : -1;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (r[j] >= 0 && r[j] < R) atomicAdd(&hist[r[j]], 1);
  }
}
template <int STEP>
__device__ __forceinline__ void write_norms(const int32_t* __restrict__ et, int beg, int end, int t,
                                            int R, const int32_t* hist,
                                            float* __restrict__ edge_norm) {
  for (int e0 = beg + t; e0 < end; e0 += 4 * STEP) {
    int r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = e0 + j * STEP < end ? et[e0 + j * STEP] : -1;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (e0 + j * STEP < end)
        edge_norm[e0 + j * STEP] = (r[j] >= 0 && r[j] < R) ? 1.0f / (float)hist[r[j]] : 0.0f;
  }
}
template <int STEP>
__device__ __forceinline__ void clear_types(const int32_t* __restrict__ et, int beg, int end, int t,
                                            int R, int32_t* hist) {
  for (int e0 = beg + t; e0 < end; e0 += 4 * STEP) {
    int r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = e0 + j * STEP < end ? et[e0 + j * STEP] : -1;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (r[j] >= 0 && r[j] < R) hist[r[j]] = 0;
  }
}

// edge_norm[e] = 1 / c(v, r_e), rows taken in the plan's degree order.  The
// long rows (the plan's split rows, perm positions 0 .. n_split - 1) are
// counted by a whole workgroup sharing one LDS histogram of R bins; every
// other row by one wave with its own.  Each pass waits for the previous one
// (a workgroup barrier, or for a wave its own LDS operations, which complete
// in issue order).
__global__ __launch_bounds__(kThreads) void k_rel_norm(const int32_t* __restrict__ rp,
                                                       const int32_t* __restrict__ et,
                                                       const int32_t* __restrict__ perm, int32_t V,
                                                       int R, float* __restrict__ edge_norm,
                                                       const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  extern __shared__ int32_t hist_all[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < (kThreads / 64) * R; i += kThreads) hist_all[i] = 0;
  __syncthreads();
  const int n_long = plan_counts[kNSplit];
  for (int64_t i = blockIdx.x; i < n_long; i += gridDim.x) {  // uniform per workgroup
    const int v = perm[i];
    const int beg = rp[v], end = rp[v + 1];
    count_types<kThreads>(et, beg, end, threadIdx.x, R, hist_all);
    __syncthreads();
    write_norms<kThreads>(et, beg, end, threadIdx.x, R, hist_all, edge_norm);
    __syncthreads();
    clear_types<kThreads>(et, beg, end, threadIdx.x, R, hist_all);
    __syncthreads();
  }
  int32_t* hist = hist_all + (int64_t)wave * R;
  const int64_t nw = (int64_t)gridDim.x * (kThreads / 64);
  for (int64_t i = n_long + (int64_t)blockIdx.x * (kThreads / 64) + wave; i < V; i += nw) {
    const int v = perm[i];
    const int beg = rp[v], end = rp[v + 1];
    count_types<64>(et, beg, end, lane, R, hist);
    lds_wait();
    write_norms<64>(et, beg, end, lane, R, hist, edge_norm);
    lds_wait();
    clear_types<64>(et, beg, end, lane, R, hist);
    lds_wait();
  }
}

// Byte flags instead of bitmap atomics (when R x W x 32 bytes is modest):
// flags[r * 32 W + u] = 1 for every (relation, source) an edge carries --
// plain byte stores of the same value, no atomics -- then packed into the
// bitmap, 32 flags per word.
__global__ __launch_bounds__(kThreads) void k_rel_flag(const int32_t* __restrict__ col,
                                                       const int32_t* __restrict__ et, int64_t E,
                                                       int R, int64_t wp,
                                                       uint8_t* __restrict__ flags,
                                                       const int32_t* __restrict__ plan_counts,
                                                       int32_t* rcounts) {
  if (plan_counts[kErrFlags]) return;
  bool bad = false;
  for (int64_t e = blockIdx.x * (int64_t)kThreads + threadIdx.x; e < E;
       e += (int64_t)gridDim.x * kThreads) {
    const int r = et[e];
    if (r < 0 || r >= R) {
      bad = true;
      continue;
    }
    uint8_t* f = flags + ((int64_t)r * wp) * 32 + col[e];
    if (*f == 0) *f = 1;
  }
  if (bad) atomicOr(&rcounts[kRelErr], 1);
}

__global__ __launch_bounds__(kThreads) void k_rel_pack(const uint8_t* __restrict__ flags,
                                                       int64_t nwords, uint32_t* __restrict__ bm,
                                                       const int32_t* __restrict__ plan_counts) {
  if (plan_counts[kErrFlags]) return;
  for (int64_t w = blockIdx.x * (int64_t)kThreads + threadIdx.x; w < nwords;
       w += (int64_t)gridDim.x * kThreads) {
    const uint4* f = reinterpret_cast<const uint4*>(flags + w * 32);
    const uint4 a = f[0], b = f[1];
    const uint32_t x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    uint32_t word = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {  // four 0/1 bytes -> four bits
      const uint32_t q = x[k];
      const uint32_t nib = (q & 1u) | ((q >> 7) & 2u) | ((q >> 14) & 4u) | ((q >> 21) & 8u);
      word |= nib << (4 * k);
    }
    bm[w] = word;
  }
}

inline unsigned grid_for(int64_t n, int64_t per, unsigned cap) {
  const int64_t g = (n + per - 1) / per;
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(g, cap));
}

}  // namespace

bool rel_layout(int32_t num_src, int64_t num_edges, int32_t num_rel, RelLayout* L) {
  if (num_src < 0 || num_edges < 0 || num_rel < 1 || num_rel > kRelMaxRelations) return false;
  const int64_t S = num_src, E = num_edges, R = num_rel;
  L->wp = std::max<int64_t>(kBlockWords, (S + 32 * kBlockWords - 1) / (32 * kBlockWords) * kBlockWords);
  L->bpr = L->wp / kBlockWords;
  L->nblocks = R * L->bpr;
  const int64_t q = std::min(E, R * S);
  int64_t mp = q + std::min(R, E) * (kRelTile - 1);
  mp = (mp + kRelTile - 1) / kRelTile * kRelTile;
  L->max_pairs = mp;
  if (mp >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return false;
  auto a256 = [](size_t x) { return (x + 255) & ~size_t(255); };
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t o = off;
    off = a256(off + n);
    return o;
  };
  L->off_rel_ptr = take((size_t)(R + 1) * 4);
  L->off_rel_count = take((size_t)R * 4);
  L->off_pair_src = take((size_t)mp * 4);
  L->off_edge_pair = take((size_t)E * 4);
  L->off_edge_norm = take((size_t)E * 4);
  L->off_counts = take(kRelCountSlots * 4);
  L->off_scratch = off;
  L->off_bitmap = take((size_t)R * L->wp * 4);
  // byte flags (32 per bitmap word) when they stay under 256 MB
  L->use_flags = (size_t)R * L->wp * 32 <= (size_t(1) << 28);
  L->off_flags = take(L->use_flags ? (size_t)R * L->wp * 32 : 0);
  L->off_word_base = take((size_t)R * L->wp * 4);
  L->off_bcnt = take((size_t)L->nblocks * 4);
  L->off_block_base = take((size_t)L->nblocks * 4);
  L->scratch_bytes = off - L->off_scratch;
  L->total = off;
  return true;
}

hipError_t launch_rel_build(const saga_plan& p, const saga_rel_plan& rel, const RelLayout& L,
                            hipStream_t st) {
  char* scratch = static_cast<char*>(rel.scratch);
  uint32_t* bm = reinterpret_cast<uint32_t*>(scratch + (L.off_bitmap - L.off_scratch));
  int32_t* word_base = reinterpret_cast<int32_t*>(scratch + (L.off_word_base - L.off_scratch));
  int32_t* bcnt = reinterpret_cast<int32_t*>(scratch + (L.off_bcnt - L.off_scratch));
  int32_t* block_base = reinterpret_cast<int32_t*>(scratch + (L.off_block_base - L.off_scratch));
  const int R = rel.num_rel;
  const int64_t E = p.num_edges;
  const int64_t nbm = (int64_t)R * L.wp;
  hipLaunchKernelGGL(k_rel_fill, dim3(1), dim3(64), 0, st, reinterpret_cast<uint32_t*>(rel.counts),
                     (int64_t)kRelCountSlots, 0u);
  if (L.use_flags) {
    uint32_t* flags = reinterpret_cast<uint32_t*>(scratch + (L.off_flags - L.off_scratch));
    hipLaunchKernelGGL(k_rel_fill, dim3(grid_for(nbm * 8, kThreads * 4, 8192)), dim3(kThreads), 0,
                       st, flags, nbm * 8, 0u);
    if (E > 0)
      hipLaunchKernelGGL(k_rel_flag, dim3(grid_for(E, kThreads * 8, 8192)), dim3(kThreads), 0, st,
                         p.col_idx, rel.etype, E, R, L.wp, reinterpret_cast<uint8_t*>(flags),
                         p.counts, rel.counts);
    hipLaunchKernelGGL(k_rel_pack, dim3(grid_for(nbm, kThreads, 8192)), dim3(kThreads), 0, st,
                       reinterpret_cast<const uint8_t*>(flags), nbm, bm, p.counts);
  } else {
    hipLaunchKernelGGL(k_rel_fill, dim3(grid_for(nbm, kThreads * 4, 4096)), dim3(kThreads), 0, st,
                       bm, nbm, 0u);
    if (E > 0)
      hipLaunchKernelGGL(k_rel_mark, dim3(grid_for(E, kThreads * 8, 8192)), dim3(kThreads), 0, st,
                         p.col_idx, rel.etype, E, R, L.wp, bm, p.counts, rel.counts);
  }
  hipLaunchKernelGGL(k_rel_bcount, dim3(grid_for(L.nblocks, 1, 8192)), dim3(kThreads), 0, st, bm,
                     L.nblocks, bcnt, p.counts);
  hipLaunchKernelGGL(k_rel_scan, dim3(1), dim3(1024), 0, st, bcnt, R, L.bpr, (int)kRelTile,
                     rel.rel_count, rel.rel_ptr, block_base, rel.counts, p.counts);
  hipLaunchKernelGGL(k_rel_pairs, dim3(grid_for(L.nblocks, 1, 8192)), dim3(kThreads), 0, st, bm,
                     L.nblocks, L.wp, block_base, word_base, rel.pair_src, p.counts);
  hipLaunchKernelGGL(k_rel_pad, dim3(grid_for(R, 1, 4096)), dim3(128), 0, st, rel.rel_ptr,
                     rel.rel_count, R, rel.pair_src, p.counts);
  if (E > 0) {
    hipLaunchKernelGGL(k_rel_edges, dim3(grid_for(E, kThreads * 8, 8192)), dim3(kThreads), 0, st,
                       p.col_idx, rel.etype, E, R, L.wp, bm, word_base, rel.edge_pair, p.counts);
    const size_t lds = (size_t)(kThreads / 64) * R * 4;
    hipLaunchKernelGGL(k_rel_norm, dim3(grid_for(p.num_dst, kThreads / 64, 16384)), dim3(kThreads),
                       lds, st, p.row_ptr, rel.etype, p.perm, p.num_dst, R, rel.edge_norm,
                       p.counts);
  }
  return hipGetLastError();
}

}  // namespace saga
