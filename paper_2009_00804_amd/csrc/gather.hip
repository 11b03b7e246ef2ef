// Fused Scatter + ApplyEdge + Gather on the in-CSR (Sec. 3.2 of the paper:
// Scatter moves the source embeddings along the edges, ApplyEdge turns them
// into messages or attention scores, Gather reduces them per destination;
// fused, the sum-Gather is the sparse adjacency x embedding product of
// Fig. 7b).  No edge tensor is materialised: every message lives only in
// registers.
//
// Work decomposition (one plan, all reductions):
//   * a "group" of LPR lanes owns one segment (<= seg_len in-edges of one
//     destination row) at a time; each lane holds a 16-byte slice of the
//     feature row (LPR = next power of two of the row's 16-byte vectors);
//   * a workgroup (256 threads) walks one row block (consecutive segments of
//     the degree-sorted order, bounded total cost), groups striding over it;
//   * the neighbour indices of a segment are read 1 per lane, coalesced, and
//     broadcast inside the group with a cross-lane permute; the source rows
//     are fetched as 128-bit loads, U rows in flight per lane;
//   * a segment that is a whole row applies the epilogue and writes the
//     output row; segments of split rows (d_in > seg_len) write float32
//     partials, merged in a fixed order by k_combine (deterministic: no
//     floating-point atomics anywhere).
#include <algorithm>
#include <utility>
#include <cstdlib>

#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kThreads = 256;
enum { kSum = 0, kMean = 1, kMax = 2, kSoftmax = 3 };

template <typename T>
__device__ __forceinline__ float load_elem(const void* p, int64_t i) {
  if constexpr (sizeof(T) == 4)
    return static_cast<const float*>(p)[i];
  else
    return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
}

// Activations other than ReLU / none, four columns per call: kept out of
// line so the transcendental code does not set the register budget of the
// gather loops that share an epilogue with it.
__device__ __noinline__ f32x4 act_slow4(int act, f32x4 v) {
  return f32x4{apply_act(act, v.x), apply_act(act, v.y), apply_act(act, v.z), apply_act(act, v.w)};
}

template <int N>
__device__ __forceinline__ void apply_act_vec(int act, float (&x)[N]) {
  if (act == SAGA_ACT_RELU) {
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] = x[i] > 0.0f ? x[i] : 0.0f;
  } else if (act != SAGA_ACT_NONE) {
#pragma unroll
    for (int i = 0; i < N; i += 4) {
      const f32x4 r = act_slow4(act, f32x4{x[i], x[i + 1], x[i + 2], x[i + 3]});
      x[i] = r.x; x[i + 1] = r.y; x[i + 2] = r.z; x[i + 3] = r.w;
    }
  }
}

// out[row, col0 .. col0 + EPV) = act(x + self + bias), clipped to out_cols
template <typename T>
__device__ __forceinline__ void store_out(const GatherArgs& a, int64_t row, int col0,
                                          float (&x)[Vec16<T>::N]) {
  constexpr int EPV = Vec16<T>::N;
  T* o = static_cast<T*>(a.out) + row * a.ld_out + col0;
  if (col0 + EPV <= a.out_cols) {
    // a whole 16-byte vector: self as one vector load (its rows are 16-byte
    // aligned), bias as EPV scalars
    if (a.self) {
      float sv[EPV];
      Vec16<T>::widen(*reinterpret_cast<const uint4*>(static_cast<const T*>(a.self) + row * a.ld_self + col0), sv);
#pragma unroll
      for (int k = 0; k < EPV; ++k) x[k] += sv[k];
    }
    if (a.bias) {
#pragma unroll
      for (int k = 0; k < EPV; ++k) x[k] += a.bias[col0 + k];
    }
    apply_act_vec(a.act, x);
    Vec16<T>::store(o, x);
  } else if (col0 < a.out_cols) {
#pragma unroll
    for (int k = 0; k < EPV; ++k) {
      const int c = col0 + k;
      float v = x[k];
      if (a.self && c < a.out_cols) v += load_elem<T>(a.self, row * a.ld_self + c);
      if (a.bias && c < a.out_cols) v += a.bias[c];
      x[k] = v;
    }
    apply_act_vec(a.act, x);
    Vec16<T>::store_n(o, x, a.out_cols - col0);
  }
}

// ------------------------------------------------------------------------
// COPY / SRC_NORM messages with SUM, MEAN or MAX
//
// Feature slicing: the row's 16-byte vectors are split into `nslices`
// slices of LPR vectors; workgroup i works on block i / nslices, slice
// i % nslices.  Workgroups are dispatched round-robin over the 8 XCDs, so
// with nslices dividing 8 every XCD touches one slice only and its L2 keeps
// nslices times more (hot) source rows than if it cached whole rows.  With
// 128-byte slices each cached line is one row's slice.
// Neighbour indices are read CPL per lane (LPR*CPL edges per batch) with
// non-temporal loads (they are streamed once) and broadcast by cross-lane
// permute; U source-row loads are kept in flight per lane.
// ------------------------------------------------------------------------
// FULL: every lane's 16-byte vector lies inside the row (the row's vectors
// are a whole number of slices), so the per-vector range checks drop out.
// O32: the source matrix spans less than 4 GiB, so a row vector's address is
// the uniform base plus a 32-bit byte offset (one register per load in
// flight instead of a 64-bit address pair).
// IDENT: the source row of edge e is row e itself (the segment reduction of
// an edge tensor already laid out in CSR order; the unfused path).
// WM: message weight -- kWNone (1), kWSrcNorm (d_out(u)^-1/2, GCN) or
// kWEdge (edge_scale[e], R-GCN's 1 / c(v, r); col_idx then holds the
// edge's pair row).
enum { kWNone = 0, kWSrcNorm = 1, kWEdge = 2 };
template <typename T, int LPR, int VPL, int U, int CPL, bool MAXRED, int WM, bool FULL,
          bool IDENT, bool O32>
__device__ __forceinline__ void gather_simple_body(const GatherArgs& a, int nslices, int slice0) {
  constexpr int EPV = Vec16<T>::N;
  constexpr int NG = kThreads / LPR;
  const int32_t* __restrict__ counts = a.counts;
  if (counts[kErrFlags]) return;
  if (WM == kWEdge && a.err2[0]) return;
  const int nb = counts[kNumBlocks];
  const int w = blockIdx.x / nslices;
  const int slice = slice0 + (blockIdx.x - w * nslices);
  const int b = w * a.bpw;  // row blocks b .. b + bpw - 1
  if (b >= nb) return;
  const int s_split = counts[kSSplit];
  const int gl = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const int gbase = (threadIdx.x & 63) - gl;
  const int nv = (int)((a.feat * (int64_t)sizeof(T) + 15) / 16);
  const int v0 = slice * LPR * VPL;
  // this lane's 16-byte vectors of every source row
  const uint4* __restrict__ src = reinterpret_cast<const uint4*>(static_cast<const T*>(a.src));
  const int64_t ld16 = a.ld_src * (int64_t)sizeof(T) / 16;
  const char* __restrict__ srcb = static_cast<const char*>(a.src);
  const uint32_t ldb = (uint32_t)(a.ld_src * (int64_t)sizeof(T));
  const int32_t* __restrict__ col = a.col_idx;
  const float init = MAXRED ? -INFINITY : 0.0f;

  const int s0 = a.block_ptr[b], s1 = a.block_ptr[b + a.bpw < nb ? b + a.bpw : nb];
  for (int s = s0 + grp; s < s1; s += NG) {
    const int row = a.seg_row[s];
    const int beg = a.seg_beg[s], end = a.seg_end[s];
    float acc[VPL][EPV];
#pragma unroll
    for (int q = 0; q < VPL; ++q)
#pragma unroll
      for (int i = 0; i < EPV; ++i) acc[q][i] = init;

    for (int e = beg; e < end; e += LPR * CPL) {
      int c[CPL];
      float cw[CPL];
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int idx = e + j * LPR + gl;
        if constexpr (IDENT)
          c[j] = idx < end ? idx : 0;
        else
          c[j] = idx < end ? __builtin_nontemporal_load(col + idx) : 0;
        if constexpr (WM == kWEdge)
          cw[j] = idx < end ? __builtin_nontemporal_load(a.edge_scale + idx) : 0.0f;
      }
      const int n = (end - e) < LPR * CPL ? (end - e) : LPR * CPL;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int nq = n - j * LPR < LPR ? n - j * LPR : LPR;
        if (nq <= 0) break;
        // U row loads in flight per lane; a short last batch is predicated
        for (int t = 0; t < nq; t += U) {
          uint4 raw[U][VPL];
          float wu[U];
#pragma unroll
          for (int k = 0; k < U; ++k) {
            const int tk = t + k < nq ? t + k : t;
            const int u = __shfl(c[j], gbase + tk, 64);
            if constexpr (WM == kWSrcNorm) wu[k] = rsqrt_deg(a.d_out[u]);
            if constexpr (WM == kWEdge) wu[k] = __shfl(cw[j], gbase + tk, 64);
#pragma unroll
            for (int q = 0; q < VPL; ++q) {
              const int vi = v0 + gl + q * LPR;
              if ((FULL || vi < nv) && t + k < nq) {
                if constexpr (O32)
                  raw[k][q] = *reinterpret_cast<const uint4*>(
                      srcb + ((uint32_t)u * ldb + (uint32_t)vi * 16u));
                else
                  raw[k][q] = src[(int64_t)u * ld16 + vi];
              }
            }
          }
#pragma unroll
          for (int k = 0; k < U; ++k) {
            if (t + k < nq) {
#pragma unroll
              for (int q = 0; q < VPL; ++q) {
                float x[EPV];
                Vec16<T>::widen(raw[k][q], x);
#pragma unroll
                for (int i = 0; i < EPV; ++i) {
                  const float v = WM != kWNone ? x[i] * wu[k] : x[i];
                  acc[q][i] = MAXRED ? fmaxf(acc[q][i], v) : acc[q][i] + v;
                }
              }
            }
          }
        }
      }
    }

    if (s < s_split) {
      // float32 partials; pstride and vi * EPV are multiples of 4 floats
      float* p = a.partial + (int64_t)s * a.pstride;
#pragma unroll
      for (int q = 0; q < VPL; ++q) {
        const int vi = v0 + gl + q * LPR;
        if (FULL || vi < nv)
#pragma unroll
          for (int i = 0; i < EPV; i += 4)
            *reinterpret_cast<f32x4*>(p + vi * EPV + i) =
                f32x4{acc[q][i], acc[q][i + 1], acc[q][i + 2], acc[q][i + 3]};
      }
    } else {
      const int d = end - beg;  // a whole row
      float scale = 1.0f;
      if (a.reduce == kMean) scale = d > 0 ? 1.0f / (float)d : 0.0f;
      if (a.dst_norm) scale *= rsqrt_deg(d);
#pragma unroll
      for (int q = 0; q < VPL; ++q) {
        const int vi = v0 + gl + q * LPR;
        if (FULL || vi < nv) {
          float x[EPV];
#pragma unroll
          for (int i = 0; i < EPV; ++i) {
            float v = acc[q][i];
            if (MAXRED && d == 0) v = 0.0f;
            x[i] = v * scale;
          }
          store_out<T>(a, row, vi * EPV, x);
        }
      }
    }
  }
}

template <typename T, int LPR, int VPL, int U, int CPL, bool MAXRED, int WM, bool FULL,
          bool IDENT = false>
__global__ __launch_bounds__(kThreads) void k_gather_simple(GatherArgs a, int nslices, int slice0) {
  gather_simple_body<T, LPR, VPL, U, CPL, MAXRED, WM, FULL, IDENT, false>(a, nslices, slice0);
}

// The plain sum over whole slices of a source below 4 GiB (the GCN Gather):
// built for eight waves per SIMD, which its registers allow without spills
// with four row loads in flight per lane (56 registers float32, 64
// bfloat16).  Measured on the 2^21 graph, 128 bfloat16 columns: 2.38 ms,
// against 2.47 with eight loads in flight at seven waves.
// FL: whole slices (else the last slice's lanes past the row are idle, as
// for 41 bfloat16 columns or the 9-column float32 tail).
template <typename T, int LPR, int VPL, int U, int CPL, bool FL = true>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(8))) void k_gather_sum(
    GatherArgs a, int nslices, int slice0) {
  gather_simple_body<T, LPR, VPL, U, CPL, false, kWNone, FL, false, true>(a, nslices, slice0);
}

// The plain max over slices of a source below 4 GiB (the GraphSAGE-pool
// Gather), built like k_gather_sum.
template <typename T, int LPR, int VPL, int U, int CPL, bool FL>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(8))) void k_gather_max(
    GatherArgs a, int nslices, int slice0) {
  gather_simple_body<T, LPR, VPL, U, CPL, true, kWNone, FL, false, true>(a, nslices, slice0);
}

// ------------------------------------------------------------------------
// The next layer's transform fused into this Gather (cross-stage
// pipelining, Sec. 4): y[v] = xrs(v) * (h_v W) for W F x xn (xn <= 64),
// h_v the finished Gather row, taken as soon as a workgroup has finished
// its rows rather than after the whole Gather.  Sixteen rows at a time go
// onto the matrix cores with the output columns as the M side (A = W^T,
// staged in LDS with k contiguous) and the rows as the N side (B = the h
// rows, read from memory with k contiguous): the k order inside a chunk is
// the same permutation on both sides, so the contraction is unchanged, and
// a lane's four accumulators are four adjacent outputs of one row.
// ------------------------------------------------------------------------
template <typename T> struct XfMma;
template <> struct XfMma<float> {
  __device__ __forceinline__ static f32x4 mma(const uint4& w, const uint4& h, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.x), __uint_as_float(h.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.y), __uint_as_float(h.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.z), __uint_as_float(h.z), c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.w), __uint_as_float(h.w), c, 0, 0, 0);
  }
};
template <> struct XfMma<uint16_t> {
  __device__ __forceinline__ static f32x4 mma(const uint4& w, const uint4& h, f32x4 c) {
    bf16x8 wa, hb;
    __builtin_memcpy(&wa, &w, 16);
    __builtin_memcpy(&hb, &h, 16);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, hb, c, 0, 0, 0);
  }
};

// one 16-row tile: lane (lr, lg) = (lane % 16, lane / 16) brings row `row`
// (-1: a padding lane of a short tile) and stores outputs 16 nt + 4 lg ..
// + 3 of it.  The rows' 64-byte chunks (at most eight: F is at most 512
// bytes) are loaded four at a time ahead of their MFMAs.
template <typename T, int NT>
__device__ __forceinline__ void xf_tile(const GatherArgs& a, int row, const uint4* wt) {
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int nk = (int)(a.feat * (int64_t)sizeof(T) / 64);
  const uint4* hp = reinterpret_cast<const uint4*>(static_cast<const T*>(a.out) +
                                                   (int64_t)(row >= 0 ? row : 0) * a.ld_out);
  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  for (int j0 = 0; j0 < nk; j0 += 4) {
    uint4 hv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      hv[j] = (row >= 0 && j0 + j < nk) ? hp[(j0 + j) * 4 + lg] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j0 + j < nk) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[nt] = XfMma<T>::mma(wt[(nt * 16 + lr) * a.xldwt + (j0 + j) * 4 + lg], hv[j], acc[nt]);
      }
    }
  }
  if (row < 0) return;
  const float rs = a.xrs ? rsqrt_deg(a.xrs[row]) : 1.0f;
  const int head = a.xsplit > 0 ? a.xsplit : a.xn;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n0 = nt * 16 + lg * 4;
    if (n0 >= a.xn) continue;
    float y[4] = {acc[nt].x * rs, acc[nt].y * rs, acc[nt].z * rs, acc[nt].w * rs};
    T* o;
    int lim;  // outputs of the four that exist (xsplit is a multiple of 4)
    if (n0 >= head) {
      o = static_cast<T*>(a.xtail) + (int64_t)row * a.ld_xtail + (n0 - head);
      lim = a.xn - n0;
    } else {
      o = static_cast<T*>(a.xout) + (int64_t)row * a.ld_xout + n0;
      lim = head - n0;
    }
    if (lim >= 4 && ((uintptr_t)o & (4 * sizeof(T) - 1)) == 0) {
      if constexpr (sizeof(T) == 4) {
        *reinterpret_cast<f32x4*>(o) = f32x4{y[0], y[1], y[2], y[3]};
      } else {
        const uint32_t lo = (uint32_t)f32_to_bf16(y[0]) | ((uint32_t)f32_to_bf16(y[1]) << 16);
        const uint32_t hi = (uint32_t)f32_to_bf16(y[2]) | ((uint32_t)f32_to_bf16(y[3]) << 16);
        *reinterpret_cast<uint2*>(o) = make_uint2(lo, hi);
      }
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (t < lim) {
          if constexpr (sizeof(T) == 4)
            o[t] = y[t];
          else
            o[t] = f32_to_bf16(y[t]);
        }
      }
    }
  }
}

// W (F x xn, row-major) -> the packed W^T of GatherArgs::xwt
template <typename T>
__global__ __launch_bounds__(kThreads) void k_xf_pack(GatherArgs a, int nrows) {
  constexpr int EPV = Vec16<T>::N;
  const int F = a.feat;
  const int per = a.xldwt * EPV;  // elements per packed row, pad included
  T* wt = reinterpret_cast<T*>(a.xwt);
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < nrows * per; i += gridDim.x * kThreads) {
    const int n = i / per, k = i - n * per;
    T v = 0;
    if (n < a.xn && k < F) v = static_cast<const T*>(a.xw)[(int64_t)k * a.xn + n];
    wt[i] = v;
  }
}

// The last slice pass of the sum Gather with the next transform fused in:
// the slice is gathered as in k_gather_sum (its part of h goes to `out`),
// then each wave multiplies the whole rows its own lane groups finished
// (lane group g of the wave takes segments s0 + 8 wave + g + 32 k; a tile
// is k = 2t, 2t + 1), whose earlier slices earlier passes wrote.  No
// workgroup barrier after the Gather: a wave whose lane groups are done
// goes on to its tiles while the others still gather.  A workgroup takes
// kXfBpw row blocks, which fills the waves' tiles better (a block averages
// about 74 rows at 2^21 vertices, 18 per wave).  Dynamic LDS: the packed
// W^T (25 KB for 128 x 41 float32, which caps the kernel at six workgroups
// per CU).
constexpr int kXfBpw = 2;
template <typename T, int U, int NT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(6))) void k_gather_sum_xf(
    GatherArgs a, int slice0) {
  extern __shared__ uint4 xf_wt[];
  const int32_t* __restrict__ counts = a.counts;
  if (counts[kErrFlags]) return;
  const int nb = counts[kNumBlocks];
  const int b = blockIdx.x * a.bpw;
  if (b >= nb) return;
  for (int i = threadIdx.x; i < NT * 16 * a.xldwt; i += kThreads) xf_wt[i] = a.xwt[i];
  __syncthreads();
  gather_simple_body<T, 8, 1, U, 4, false, kWNone, true, false, true>(a, 1, slice0);
  // the lanes of this wave read rows other lanes of it stored
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  const int s_split = counts[kSSplit];
  const int s0 = a.block_ptr[b], s1 = a.block_ptr[b + a.bpw < nb ? b + a.bpw : nb];
  const int wave = threadIdx.x >> 6, lr = threadIdx.x & 15;
  constexpr int NG = kThreads / 8;  // lane groups of the workgroup
  for (int t0 = s0 + wave * 8; t0 < s1; t0 += 2 * NG) {
    const int s = t0 + (lr & 7) + (lr >> 3) * NG;
    xf_tile<T, NT>(a, s < s1 && s >= s_split ? a.seg_row[s] : -1, xf_wt);
  }
}

// The transform of the split rows (perm positions 0 .. n_split - 1), whose
// h rows k_combine has just finished.
template <typename T, int NT>
__global__ __launch_bounds__(kThreads) void k_xf_rows(GatherArgs a) {
  extern __shared__ uint4 xf_wt[];
  const int32_t* __restrict__ counts = a.counts;
  if (counts[kErrFlags]) return;
  const int n_split = counts[kNSplit];
  if (blockIdx.x * (kThreads / 4) >= n_split) return;
  for (int i = threadIdx.x; i < NT * 16 * a.xldwt; i += kThreads) xf_wt[i] = a.xwt[i];
  __syncthreads();
  const int wave = threadIdx.x >> 6, lr = threadIdx.x & 15;
  for (int t0 = (blockIdx.x * (kThreads / 64) + wave) * 16; t0 < n_split;
       t0 += gridDim.x * (kThreads / 4)) {
    const int i = t0 + lr;
    xf_tile<T, NT>(a, i < n_split ? a.perm[i] : -1, xf_wt);
  }
}

// ------------------------------------------------------------------------
// Unfused Scatter + ApplyEdge (the baseline of Fig. 7a): materialise the
// edge tensor msg[e] = w(u) * src[u] for every edge e = (u -> v) in CSR
// order, w(u) = d_out(u)^-1/2 for the GCN source norm, else 1.  One thread
// per 16-byte vector; the lanes of a row are consecutive, so both the row
// read and the message write are contiguous.
// ------------------------------------------------------------------------
template <typename T, bool SRCNORM>
__global__ __launch_bounds__(kThreads) void k_index_select(const int32_t* __restrict__ col,
                                                           int64_t E, int nv,
                                                           const uint4* __restrict__ src,
                                                           int64_t ld16,
                                                           const int32_t* __restrict__ d_out,
                                                           uint4* __restrict__ msg, int64_t ldm16,
                                                           const int32_t* __restrict__ counts) {
  if (counts[kErrFlags]) return;
  const int64_t total = E * nv;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t e = i / nv;
    const int v = (int)(i - e * nv);
    const int32_t u = col[e];
    uint4 r = src[(int64_t)u * ld16 + v];
    if constexpr (SRCNORM) {
      float x[Vec16<T>::N];
      Vec16<T>::widen(r, x);
      const float w = rsqrt_deg(d_out[u]);
#pragma unroll
      for (int k = 0; k < Vec16<T>::N; ++k) x[k] *= w;
      if constexpr (sizeof(T) == 4) {
        r = make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                       __float_as_uint(x[3]));
      } else {
        uint32_t w4[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          w4[k] = (uint32_t)f32_to_bf16(x[2 * k]) | ((uint32_t)f32_to_bf16(x[2 * k + 1]) << 16);
        r = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }
    }
    msg[e * ldm16 + v] = r;
  }
}

// ------------------------------------------------------------------------
// GAT: LeakyReLU(el[u] + er[v]) scores, online softmax per head (float32)
// ------------------------------------------------------------------------
template <int LPR, int U>
__global__ __launch_bounds__(kThreads) void k_gather_gat(GatherArgs a) {
  constexpr int NG = kThreads / LPR;
  const int32_t* __restrict__ counts = a.counts;
  if (counts[kErrFlags]) return;
  const int nb = counts[kNumBlocks];
  const int s_split = counts[kSSplit];
  const int gl = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const int gbase = (threadIdx.x & 63) - gl;
  const int F = a.feat, H = a.heads, D = F / H;
  const int nv = F / 4;
  const bool active = gl < nv;
  const int head = active ? (gl * 4) / D : 0;
  const float* __restrict__ z = static_cast<const float*>(a.src);
  const int32_t* __restrict__ col = a.col_idx;
  const float slope = a.neg_slope;

  for (int b = blockIdx.x * a.bpw; b < nb; b += gridDim.x * a.bpw) {
    const int s0 = a.block_ptr[b], s1 = a.block_ptr[b + a.bpw < nb ? b + a.bpw : nb];
    for (int s = s0 + grp; s < s1; s += NG) {
      const int row = a.seg_row[s];
      const int beg = a.seg_beg[s], end = a.seg_end[s];
      const float erv = active ? a.er[(int64_t)row * a.ld_er + head] : 0.0f;
      float m = -INFINITY, l = 0.0f;
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int e = beg; e < end; e += LPR) {
        const int my = e + gl;
        const int c = my < end ? col[my] : 0;
        const int n = (end - e) < LPR ? (end - e) : LPR;
        for (int t = 0; t < n; t += U) {
          int u[U];
          float sc[U], x[U][4];
#pragma unroll
          for (int k = 0; k < U; ++k) {
            u[k] = __shfl(c, gbase + ((t + k) < n ? t + k : t), 64);
            if (active) {
              sc[k] = a.el[(int64_t)u[k] * a.ld_el + head];
              Vec16<float>::load(z + (int64_t)u[k] * a.ld_src + gl * 4, x[k]);
            }
          }
#pragma unroll
          for (int k = 0; k < U; ++k) {
            if (t + k < n) {
              float sv = sc[k] + erv;
              sv = sv > 0.0f ? sv : slope * sv;
              const float mn = fmaxf(m, sv);
              const float f = __expf(m - mn);
              const float p = __expf(sv - mn);
              l = l * f + p;
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[i] = acc[i] * f + p * x[k][i];
              m = mn;
            }
          }
        }
      }
      if (s < s_split) {
        if (active) {
          float* p = a.partial + (int64_t)s * a.pstride;
#pragma unroll
          for (int i = 0; i < 4; ++i) p[gl * 4 + i] = acc[i];
          if ((gl * 4) % D == 0) {
            p[a.pcols + head] = m;
            p[a.pcols + H + head] = l;
          }
        }
      } else {
        float o[4];
        const float inv = l > 0.0f ? 1.0f / l : 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = active ? acc[i] * inv : 0.0f;
        if (a.head_mean) {
          // sum over heads: lanes gl = head * (D/4) + off
          for (int k = D / 4; k < nv; k <<= 1)
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] += __shfl_xor(o[i], k, 64);
          if (active && head == 0) {
            const float r = 1.0f / (float)H;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] *= r;
            store_out<float>(a, row, gl * 4, o);
          }
        } else if (active) {
          store_out<float>(a, row, gl * 4, o);
        }
      }
    }
  }
}

// ------------------------------------------------------------------------
// Gated messages: sigmoid(gs[u] + gd[v] + b_e + e_uv W_ee) * h[u], SUM
// (float32, F = 64, one 16-byte slice of 4 features per lane)
// ------------------------------------------------------------------------
// pre += sum_j e_j W[j][4 columns of this lane], e_j held by lane j of the
// lane's 16-lane group: ds_swizzle in bit mode reads lane (lane & 16) | j of
// each 32-lane half, i.e. lane j of the group (every lane takes part)
template <int J>
__device__ __forceinline__ void project_one(float ev, const float (&wr)[16][4], float (&pre)[4]) {
  const float ej = __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(ev), 0x10 | (J << 5)));
#pragma unroll
  for (int q = 0; q < 4; ++q) pre[q] += ej * wr[J][q];
}
template <int... J>
__device__ __forceinline__ void project_edge(float ev, const float (&wr)[16][4], float (&pre)[4],
                                             std::integer_sequence<int, J...>) {
  (project_one<J>(ev, wr, pre), ...);
}

template <int LPR, int U>
__global__ __launch_bounds__(kThreads) void k_gather_gated(GatherArgs a) {
  static_assert(LPR == 16, "the edge-feature broadcast works on 16-lane groups");
  constexpr int NG = kThreads / LPR;
  constexpr int FE_MAX = 16;
  const int32_t* __restrict__ counts = a.counts;
  if (counts[kErrFlags]) return;
  const int nb = counts[kNumBlocks];
  const int s_split = counts[kSSplit];
  const int gl = threadIdx.x % LPR;
  const int grp = threadIdx.x / LPR;
  const int gbase = (threadIdx.x & 63) - gl;
  const int F = a.feat, Fe = a.fe;
  const int nv = F / 4;
  const bool active = gl < nv;
  const float* __restrict__ h = static_cast<const float*>(a.src);
  const int32_t* __restrict__ col = a.col_idx;
  float wr[FE_MAX][4];
#pragma unroll
  for (int i = 0; i < FE_MAX; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      wr[i][q] = (active && i < Fe) ? a.w_edge[(int64_t)i * F + gl * 4 + q] : 0.0f;
  float gb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) gb[q] = (active && a.gate_bias) ? a.gate_bias[gl * 4 + q] : 0.0f;

  for (int b = blockIdx.x * a.bpw; b < nb; b += gridDim.x * a.bpw) {
    const int s0 = a.block_ptr[b], s1 = a.block_ptr[b + a.bpw < nb ? b + a.bpw : nb];
    for (int s = s0 + grp; s < s1; s += NG) {
      const int row = a.seg_row[s];
      const int beg = a.seg_beg[s], end = a.seg_end[s];
      float gd[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if (active) {
        Vec16<float>::load(a.gdst + (int64_t)row * a.ld_gdst + gl * 4, gd);
#pragma unroll
        for (int q = 0; q < 4; ++q) gd[q] += gb[q];
      }
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int e = beg; e < end; e += LPR) {
        const int my = e + gl;
        const int c = my < end ? col[my] : 0;
        const int n = (end - e) < LPR ? (end - e) : LPR;
        // U edges' loads (h_u, S_src[u], e_uv) in flight before the math;
        // a short last batch repeats its first edge and skips it
        for (int t = 0; t < n; t += U) {
          // e_uv: lane j of the group holds feature j (one coalesced row
          // load per edge), broadcast to the group inside the projection
          float hs[U][4], gs[U][4], ev[U];
#pragma unroll
          for (int k = 0; k < U; ++k) {
            const int tk = t + k < n ? t + k : t;
            const int u = __shfl(c, gbase + tk, 64);
            ev[k] = gl < Fe ? a.efeat[(int64_t)(e + tk) * a.ld_efeat + gl] : 0.0f;
            if (active) {
              Vec16<float>::load(h + (int64_t)u * a.ld_src + gl * 4, hs[k]);
              Vec16<float>::load(a.gsrc + (int64_t)u * a.ld_gsrc + gl * 4, gs[k]);
            }
          }
#pragma unroll
          for (int k = 0; k < U; ++k) {
            float pre[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) pre[q] = gs[k][q] + gd[q];
            project_edge(ev[k], wr, pre, std::make_integer_sequence<int, FE_MAX>{});
            if (active && t + k < n) {
#pragma unroll
              for (int q = 0; q < 4; ++q) acc[q] += sigmoidf_(pre[q]) * hs[k][q];
            }
          }
        }
      }
      if (!active) continue;
      if (s < s_split) {
        float* p = a.partial + (int64_t)s * a.pstride;
#pragma unroll
        for (int q = 0; q < 4; ++q) p[gl * 4 + q] = acc[q];
      } else {
        store_out<float>(a, row, gl * 4, acc);
      }
    }
  }
}

// ------------------------------------------------------------------------
// Split rows: merge the segment partials of each row.  The result does not
// depend on timing: every merge follows a fixed order or a fixed tree.
//  - Edge softmax: thread t handles column t % pc of every SPL-th segment;
//    the SPL partial results are then merged in order through LDS.
//  - Sum, mean and max, the first kCombineWgRows split rows (the longest:
//    rows are in degree order): the workgroup deals the row's segments
//    round-robin to groups of pc / 4 lanes, each lane holding four columns,
//    and the groups' values are merged in group order through LDS.
//  - Sum, mean and max, the other split rows: one wave per row, no barrier,
//    so that many rows are in flight per CU; the lanes' values are merged by
//    a fixed shuffle tree.
// ------------------------------------------------------------------------
constexpr int kCombineWgRows = 256;

__device__ __forceinline__ void merge4(int red, float4& A, const float4& x) {
  if (red == kMax) {
    A.x = fmaxf(A.x, x.x); A.y = fmaxf(A.y, x.y);
    A.z = fmaxf(A.z, x.z); A.w = fmaxf(A.w, x.w);
  } else {
    A.x += x.x; A.y += x.y; A.z += x.z; A.w += x.w;
  }
}

// the merged value of one output column of a split row: reduction finish,
// then the self term, bias and activation, stored
template <typename T>
__device__ __forceinline__ void combine_store(const GatherArgs& a, int row, int d, int c, float v) {
  const int red = a.reduce;
  if (red == kMax && d == 0) v = 0.0f;
  if (red == kMean) v = d > 0 ? v / (float)d : 0.0f;
  if (a.dst_norm) v *= rsqrt_deg(d);
  if (a.self) v += load_elem<T>(a.self, (int64_t)row * a.ld_self + c);
  if (a.bias) v += a.bias[c];
  v = apply_act(a.act, v);
  T* o = static_cast<T*>(a.out) + (int64_t)row * a.ld_out + c;
  if constexpr (sizeof(T) == 4)
    *o = v;
  else
    *o = f32_to_bf16(v);
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_combine(GatherArgs a) {
  __shared__ float sm_acc[kThreads];
  __shared__ float sm_m[kThreads];
  __shared__ float sm_l[kThreads];
  __shared__ float fin[1024];
  __shared__ float4 sm4[kThreads];
  const int32_t* __restrict__ counts = a.counts;
  if (counts[kErrFlags]) return;
  if (a.err2 && a.err2[0]) return;
  const int n_split = counts[kNSplit];
  const int red = a.reduce;
  const int F = a.feat;
  const int pc = a.pcols;  // partial columns (F rounded up to 8), <= 1024
  const int H = a.heads > 0 ? a.heads : 1;
  const int D = F / H;
  const int spl = pc >= kThreads ? 1 : kThreads / pc;
  const int t = threadIdx.x;

  if (red == kSoftmax) {
    for (int i = blockIdx.x; i < n_split; i += gridDim.x) {
      const int row = a.perm[i];
      const int f0 = a.row_seg_first[i], f1 = a.row_seg_first[i + 1];
      const int d = a.d_in[row];
      for (int c0 = 0; c0 < pc; c0 += kThreads) {
        int colc, sp;
        bool on;
        if (spl > 1) {
          sp = t / pc;
          colc = t % pc;
          on = sp < spl;
        } else {
          sp = 0;
          colc = c0 + t;
          on = colc < pc;
        }
        float A = red == kMax ? -INFINITY : 0.0f, M = -INFINITY, L = 0.0f;
        if (on) {
          const int hd = (red == kSoftmax && colc < F) ? colc / D : 0;
          // partial j merged into (A, M, L); the order of j is kept
          auto merge = [&](float v, float mj, float lj) {
            if (red == kMax) {
              A = fmaxf(A, v);
            } else if (red == kSoftmax) {
              const float mn = fmaxf(M, mj);
              const float fa = __expf(M - mn), fb = __expf(mj - mn);
              A = A * fa + v * fb;
              L = L * fa + lj * fb;
              M = mn;
            } else {
              A += v;
            }
          };
          // a hub row has hundreds of segments: UJ of its partials are read
          // before any is merged, so their loads overlap
          constexpr int UJ = 8;
          int j = f0 + sp;
          for (; j + (UJ - 1) * spl < f1; j += UJ * spl) {
            float v[UJ], mj[UJ], lj[UJ];
  #pragma unroll
            for (int u = 0; u < UJ; ++u) {
              const float* p = a.partial + (int64_t)(j + u * spl) * a.pstride;
              v[u] = p[colc];
              mj[u] = red == kSoftmax ? p[pc + hd] : 0.0f;
              lj[u] = red == kSoftmax ? p[pc + H + hd] : 0.0f;
            }
  #pragma unroll
            for (int u = 0; u < UJ; ++u) merge(v[u], mj[u], lj[u]);
          }
          for (; j < f1; j += spl) {
            const float* p = a.partial + (int64_t)j * a.pstride;
            merge(p[colc], red == kSoftmax ? p[pc + hd] : 0.0f, red == kSoftmax ? p[pc + H + hd] : 0.0f);
          }
        }
        sm_acc[t] = A;
        sm_m[t] = M;
        sm_l[t] = L;
        __syncthreads();
        if (on && sp == 0) {
          for (int q = 1; q < spl; ++q) {
            const int o = q * pc + colc;
            if (red == kMax) {
              A = fmaxf(A, sm_acc[o]);
            } else if (red == kSoftmax) {
              const float mn = fmaxf(M, sm_m[o]);
              const float fa = __expf(M - mn), fb = __expf(sm_m[o] - mn);
              A = A * fa + sm_acc[o] * fb;
              L = L * fa + sm_l[o] * fb;
              M = mn;
            } else {
              A += sm_acc[o];
            }
          }
          float v;
          if (red == kSoftmax) {
            v = L > 0.0f ? A / L : 0.0f;
          } else {
            v = A;
            if (red == kMax && d == 0) v = 0.0f;
            if (red == kMean) v = d > 0 ? v / (float)d : 0.0f;
            if (a.dst_norm) v *= rsqrt_deg(d);
          }
          fin[colc] = v;
        }
        __syncthreads();
      }
      // epilogue over output columns
      for (int c = t; c < a.out_cols; c += kThreads) {
        float v;
        if (a.head_mean) {
          v = 0.0f;
          for (int k = 0; k < H; ++k) v += fin[k * D + c];
          v *= 1.0f / (float)H;
        } else {
          v = fin[c];
        }
        if (a.self) v += load_elem<T>(a.self, (int64_t)row * a.ld_self + c);
        if (a.bias) v += a.bias[c];
        v = apply_act(a.act, v);
        T* o = static_cast<T*>(a.out) + (int64_t)row * a.ld_out + c;
        if constexpr (sizeof(T) == 4)
          *o = v;
        else
          *o = f32_to_bf16(v);
      }
      __syncthreads();
    }
    return;
  }

  // sum, mean, max; a partial row is vpr 16-byte vectors
  const int vpr = pc / 4;
  const float init = red == kMax ? -INFINITY : 0.0f;
  constexpr int UJ = 8;  // partials read before any is merged, so that loads overlap
  const int nwg = n_split < kCombineWgRows ? n_split : kCombineWgRows;
  {  // the longest rows: a whole workgroup each
    const int ng = kThreads / vpr;
    const int vg = t / vpr, vv = t % vpr;
    for (int i = blockIdx.x; i < nwg; i += gridDim.x) {
      const int row = a.perm[i];
      const int f0 = a.row_seg_first[i], f1 = a.row_seg_first[i + 1];
      const int d = a.d_in[row];
      float4 A = make_float4(init, init, init, init);
      if (vg < ng) {
        int j = f0 + vg;
        for (; j + (UJ - 1) * ng < f1; j += UJ * ng) {
          float4 x[UJ];
#pragma unroll
          for (int u = 0; u < UJ; ++u)
            x[u] = *reinterpret_cast<const float4*>(a.partial + (int64_t)(j + u * ng) * a.pstride +
                                                    4 * vv);
#pragma unroll
          for (int u = 0; u < UJ; ++u) merge4(red, A, x[u]);
        }
        for (; j < f1; j += ng)
          merge4(red, A, *reinterpret_cast<const float4*>(a.partial + (int64_t)j * a.pstride + 4 * vv));
      }
      sm4[t] = A;
      __syncthreads();
      if (vg == 0) {
        for (int q = 1; q < ng; ++q) merge4(red, A, sm4[q * vpr + vv]);
        const float r[4] = {A.x, A.y, A.z, A.w};
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (4 * vv + k < a.out_cols) combine_store<T>(a, row, d, 4 * vv + k, r[k]);
      }
      __syncthreads();
    }
  }
  {  // the other rows: one wave each.  With vpr < 64 a wave instruction
     // covers spw segments (lane = sub * vpr + vector); otherwise the
     // vectors are taken 64 at a time.
    const int lane = t & 63;
    const int spw = vpr >= 64 ? 1 : 64 / vpr;
    const int sub = vpr >= 64 ? 0 : lane / vpr;
    const int waves = kThreads / 64;
    for (int i = nwg + blockIdx.x * waves + (t >> 6); i < n_split; i += gridDim.x * waves) {
      const int row = a.perm[i];
      const int f0 = a.row_seg_first[i], f1 = a.row_seg_first[i + 1];
      const int d = a.d_in[row];
      for (int v0 = 0; v0 < vpr; v0 += 64) {
        const int vv = vpr >= 64 ? v0 + lane : lane % vpr;
        const bool on = sub < spw && vv < vpr;
        float4 A = make_float4(init, init, init, init);
        if (on) {
          int j = f0 + sub;
          for (; j + (UJ - 1) * spw < f1; j += UJ * spw) {
            float4 x[UJ];
#pragma unroll
            for (int u = 0; u < UJ; ++u)
              x[u] = *reinterpret_cast<const float4*>(a.partial +
                                                      (int64_t)(j + u * spw) * a.pstride + 4 * vv);
#pragma unroll
            for (int u = 0; u < UJ; ++u) merge4(red, A, x[u]);
          }
          for (; j < f1; j += spw)
            merge4(red, A, *reinterpret_cast<const float4*>(a.partial + (int64_t)j * a.pstride + 4 * vv));
        }
        // tree over the subs: at step s, sub k (k % 2s == 0) takes sub k + s
        for (int s = 1; s < spw; s <<= 1) {
          const int src = lane + s * vpr;
          float4 y;
          y.x = __shfl(A.x, src < 64 ? src : lane, 64);
          y.y = __shfl(A.y, src < 64 ? src : lane, 64);
          y.z = __shfl(A.z, src < 64 ? src : lane, 64);
          y.w = __shfl(A.w, src < 64 ? src : lane, 64);
          if (sub % (2 * s) == 0 && sub + s < spw) merge4(red, A, y);
        }
        if (on && sub == 0) {
          const float r[4] = {A.x, A.y, A.z, A.w};
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (4 * vv + k < a.out_cols) combine_store<T>(a, row, d, 4 * vv + k, r[k]);
        }
      }
    }
  }
}

__global__ void k_fold_attention(const float* __restrict__ w, int64_t K, int64_t F, int H,
                                 const float* __restrict__ al, const float* __restrict__ ar,
                                 float* __restrict__ wx, int64_t ldx) {
  const int64_t ncol = F + 2 * H;
  const int64_t n = K * ncol;
  const int64_t D = F / H;
  for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = idx / ncol, c = idx % ncol;
    float v;
    if (c < F) {
      v = w[k * F + c];
    } else {
      const int64_t hh = (c - F) % H;
      const float* att = (c - F) < H ? al : ar;
      v = 0.0f;
      for (int64_t dd = 0; dd < D; ++dd) v += w[k * F + hh * D + dd] * att[hh * D + dd];
    }
    wx[k * ldx + c] = v;
  }
}

inline int next_pow2(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Slices processed concurrently by one launch; the rest run as further
// launches.  The source rows one launch touches (src_rows x the slices'
// bytes) are kept within 192 MB, under the 256 MB Infinity Cache: on the
// 2^21-row source one 128-byte slice per launch (268 MB) measured fastest,
// while a source of 131,072 rows has all eight 128-byte slices of its
// 1 KB rows in one launch (134 MB), which also spares the launches their
// ramp and tail.  A sweep build (SAGA_SWEEP_BUILD) reads an override from
// SAGA_GATHER_CONCURRENT_SLICES (0 = all in one launch); the library itself
// reads no environment.
constexpr int64_t kSliceBudget = int64_t(192) << 20;

int concurrent_slices(const GatherArgs& a, int nslices, int slice_bytes_) {
#ifdef SAGA_SWEEP_BUILD
  static int env = [] {
    const char* e = getenv("SAGA_GATHER_CONCURRENT_SLICES");
    return e ? atoi(e) : -1;
  }();
  if (env >= 0) return env;
#endif
  const int64_t per = std::max<int64_t>(1, a.src_rows) * slice_bytes_;
  int c = 1;
  for (int k = nslices; k >= 1; --k)
    if (nslices % k == 0 && k * per <= kSliceBudget) {
      c = k;
      break;
    }
  return c;
}

template <typename T, int LPR, int VPL>
hipError_t launch_simple_lpr(const GatherArgs& a, unsigned blocks, int nslices, hipStream_t st) {
  // row loads in flight per lane: bfloat16 rows of one 16-byte vector per
  // lane keep eight in flight (the narrow layer-2 Gather: 1.45 against 1.58
  // ms with four); the sliced sum (k_gather_sum, built for eight waves per
  // SIMD) keeps four
  constexpr int U = LPR >= 8 ? (VPL == 1 && sizeof(T) == 2 ? 8 : 4) : LPR;
  constexpr int US = LPR >= 8 ? 4 : LPR;
  constexpr int CPL = LPR >= 32 ? 1 : (LPR >= 8 ? 4 : 8);
  int conc = concurrent_slices(a, nslices, LPR * VPL * 16);
  if (conc <= 0 || conc > nslices || nslices % conc != 0) conc = nslices;
  const dim3 grid(blocks * conc);
  const bool srcnorm = a.msg == SAGA_MSG_SRC_NORM;
  const int nv = (int)((a.feat * (int64_t)sizeof(T) + 15) / 16);
  const bool full = nv == nslices * LPR * VPL;
  // every row a valid column index can name lies within 4 GiB of the base
  const bool o32 = a.src_rows * a.ld_src * (int64_t)sizeof(T) <= (int64_t(1) << 32);
  for (int s0 = 0; s0 < nslices; s0 += conc) {
#define SAGA_LAUNCH(MX, WM, FL)                                                              \
  hipLaunchKernelGGL((k_gather_simple<T, LPR, VPL, U, CPL, MX, WM, FL>), grid, dim3(kThreads), \
                     0, st, a, conc, s0)
#define SAGA_LAUNCH_FULL(MX, WM)   \
  do {                             \
    if (full)                      \
      SAGA_LAUNCH(MX, WM, true);   \
    else                           \
      SAGA_LAUNCH(MX, WM, false);  \
  } while (0)
#define SAGA_LAUNCH_IDENT(MX)                                                                  \
  hipLaunchKernelGGL((k_gather_simple<T, LPR, VPL, U, CPL, MX, kWNone, false, true>), grid,    \
                     dim3(kThreads), 0, st, a, conc, s0)
    if (a.identity) {
      if (a.reduce == kMax) SAGA_LAUNCH_IDENT(true);
      else SAGA_LAUNCH_IDENT(false);
    } else if (a.msg == SAGA_MSG_TYPED) {
      SAGA_LAUNCH_FULL(false, kWEdge);
    } else if (a.reduce == kMax) {
      if (srcnorm) {
        SAGA_LAUNCH_FULL(true, kWSrcNorm);
      } else if (LPR <= 8 && o32) {
        if constexpr (LPR <= 8) {
          if (full)
            hipLaunchKernelGGL((k_gather_max<T, LPR, VPL, US, CPL, true>), grid, dim3(kThreads), 0,
                               st, a, conc, s0);
          else
            hipLaunchKernelGGL((k_gather_max<T, LPR, VPL, US, CPL, false>), grid, dim3(kThreads), 0,
                               st, a, conc, s0);
        }
      } else {
        SAGA_LAUNCH_FULL(true, kWNone);
      }
    } else if (srcnorm) {
      SAGA_LAUNCH_FULL(false, kWSrcNorm);
    } else if (LPR <= 8 && o32) {
      // (slices of at most 128 bytes: wider lane groups never take this
      // path with 128-byte slices, and are not built)
      if constexpr (LPR <= 8) {
        if (full)
          hipLaunchKernelGGL((k_gather_sum<T, LPR, VPL, US, CPL, true>), grid, dim3(kThreads), 0, st,
                             a, conc, s0);
        else
          hipLaunchKernelGGL((k_gather_sum<T, LPR, VPL, US, CPL, false>), grid, dim3(kThreads), 0,
                             st, a, conc, s0);
      }
    } else {
      SAGA_LAUNCH_FULL(false, kWNone);
    }
#undef SAGA_LAUNCH
#undef SAGA_LAUNCH_FULL
#undef SAGA_LAUNCH_IDENT
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Row blocks each workgroup takes: small blocks are paired up until a
// workgroup holds about 2048 cost units, as long as 1024 workgroups remain.
// Measured: the SAGE-pool max Gather (1024-cost blocks, eight 128-byte
// slices in one launch) runs 23 % faster two blocks to a workgroup, the
// gated layer 3 % faster; 2048- and 4096-cost blocks (R-GCN, the 2^21 GCN)
// run fastest alone, and the GAT graph's 1185 blocks would leave CUs idle.
// A sweep build reads an override from SAGA_GATHER_BLOCKS_PER_WG.
int blocks_per_wg(const GatherArgs& a) {
#ifdef SAGA_SWEEP_BUILD
  static int env = [] {
    const char* e = getenv("SAGA_GATHER_BLOCKS_PER_WG");
    int x = e ? atoi(e) : 0;
    return x >= 1 && x <= 64 ? x : 0;
  }();
  if (env) return env;
#endif
  int k = 1;
  while (2 * k * (int64_t)a.block_cost <= 2048 && a.max_blocks / (2 * k) >= 1024) k *= 2;
  return k;
}

// bytes of each source row one slice covers: 128, one L2 line (a sweep
// build reads other widths from SAGA_GATHER_SLICE_BYTES)
#ifdef SAGA_SWEEP_BUILD
int slice_bytes() {
  static int v = [] {
    const char* e = getenv("SAGA_GATHER_SLICE_BYTES");
    int x = e ? atoi(e) : 128;
    return x >= 16 ? x : 128;
  }();
  return v;
}
#else
constexpr int slice_bytes() { return 128; }
#endif

template <typename T>
hipError_t launch_simple(const GatherArgs& a, int nv, unsigned blocks, hipStream_t st) {
  const int sv = slice_bytes() / 16;
  if (sv >= 1 && nv > sv && nv % sv == 0 && (sv & (sv - 1)) == 0 && sv <= 64) {
    const int ns = nv / sv;
#ifndef SAGA_SWEEP_BUILD
    return launch_simple_lpr<T, 8, 1>(a, blocks, ns, st);
#else
    switch (sv) {
      case 1: return launch_simple_lpr<T, 1, 1>(a, blocks, ns, st);
      case 2: return launch_simple_lpr<T, 2, 1>(a, blocks, ns, st);
      case 4: return launch_simple_lpr<T, 4, 1>(a, blocks, ns, st);
      case 8: return launch_simple_lpr<T, 8, 1>(a, blocks, ns, st);
      case 16: return launch_simple_lpr<T, 16, 1>(a, blocks, ns, st);
      case 32: return launch_simple_lpr<T, 32, 1>(a, blocks, ns, st);
      default: return launch_simple_lpr<T, 64, 1>(a, blocks, ns, st);
    }
#endif
  }
  // rows past 2 KB (64 lanes x 2 vectors): 128-byte slices, the last one
  // ragged (its lanes past the row end load nothing)
  if (nv > 128) return launch_simple_lpr<T, 8, 1>(a, blocks, (nv + 7) / 8, st);
  if (nv > 64) return launch_simple_lpr<T, 64, 2>(a, blocks, 1, st);
  switch (next_pow2(nv)) {
    case 1: return launch_simple_lpr<T, 1, 1>(a, blocks, 1, st);
    case 2: return launch_simple_lpr<T, 2, 1>(a, blocks, 1, st);
    case 4: return launch_simple_lpr<T, 4, 1>(a, blocks, 1, st);
    case 8: return launch_simple_lpr<T, 8, 1>(a, blocks, 1, st);
    case 16: return launch_simple_lpr<T, 16, 1>(a, blocks, 1, st);
    case 32: return launch_simple_lpr<T, 32, 1>(a, blocks, 1, st);
    default: return launch_simple_lpr<T, 64, 1>(a, blocks, 1, st);
  }
}

}  // namespace

int gather_partial_cols(int64_t feat) { return (int)((feat + 7) / 8 * 8); }

size_t gather_partial_stride(const saga_edge_op& op, int64_t feat) {
  int64_t pc = gather_partial_cols(feat);
  if (op.reduce == SAGA_RED_SOFTMAX) pc += 2 * op.heads;
  return (size_t)((pc + 3) / 4 * 4);
}

hipError_t launch_gather(const GatherArgs& a0, hipStream_t st) {
  GatherArgs a = a0;
  a.bpw = blocks_per_wg(a);
  const unsigned grid = (unsigned)(a.max_blocks > 0 ? (a.max_blocks + a.bpw - 1) / a.bpw : 1);
  const int esz = a.dtype == SAGA_BF16 ? 2 : 4;
  const int nv = (int)((a.feat * (int64_t)esz + 15) / 16);
  hipError_t err = hipSuccess;
  if (a.msg == SAGA_MSG_GAT) {
    const int lpr = next_pow2(nv);
    switch (lpr) {
      case 1: hipLaunchKernelGGL((k_gather_gat<1, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
      case 2: hipLaunchKernelGGL((k_gather_gat<2, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
      case 4: hipLaunchKernelGGL((k_gather_gat<4, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
      case 8: hipLaunchKernelGGL((k_gather_gat<8, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
      case 16: hipLaunchKernelGGL((k_gather_gat<16, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
      case 32: hipLaunchKernelGGL((k_gather_gat<32, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
      default: hipLaunchKernelGGL((k_gather_gat<64, 4>), dim3(grid), dim3(kThreads), 0, st, a); break;
    }
    err = hipGetLastError();
  } else if (a.msg == SAGA_MSG_GATED) {
    hipLaunchKernelGGL((k_gather_gated<16, 4>), dim3(grid), dim3(kThreads), 0, st, a);
    err = hipGetLastError();
  } else if (a.dtype == SAGA_BF16) {
    err = launch_simple<uint16_t>(a, nv, grid, st);
  } else {
    err = launch_simple<float>(a, nv, grid, st);
  }
  if (err != hipSuccess) return err;
  if (a.max_split > 0) {
    const unsigned cg = (unsigned)(a.max_split < 4096 ? a.max_split : 4096);
    if (a.dtype == SAGA_BF16)
      hipLaunchKernelGGL(k_combine<uint16_t>, dim3(cg), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(k_combine<float>, dim3(cg), dim3(kThreads), 0, st, a);
    err = hipGetLastError();
  }
  return err;
}

int64_t xf_pack_bytes(int64_t feat, int esize, int xn) {
  return (int64_t)(xn + 15) / 16 * 16 * (feat * esize / 16 + 1) * 16;
}

namespace {

template <typename T, int NT>
hipError_t launch_xf(const GatherArgs& a, unsigned grid, int nslices, hipStream_t st) {
  const size_t lds = (size_t)NT * 16 * a.xldwt * 16;
  const unsigned pb = (unsigned)((NT * 16 * a.xldwt * Vec16<T>::N + kThreads - 1) / kThreads);
  hipLaunchKernelGGL((k_xf_pack<T>), dim3(pb), dim3(kThreads), 0, st, a, NT * 16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the earlier slices, one launch each; U as in the plain sliced Gather
  constexpr int U = 4;
  for (int s0 = 0; s0 < nslices - 1; ++s0) {
    hipLaunchKernelGGL((k_gather_sum<T, 8, 1, U, 4>), dim3(grid), dim3(kThreads), 0, st, a, 1, s0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  GatherArgs ax = a;
  ax.bpw = a.bpw * kXfBpw;
  const unsigned gx = (unsigned)(a.max_blocks > 0 ? (a.max_blocks + ax.bpw - 1) / ax.bpw : 1);
  hipLaunchKernelGGL((k_gather_sum_xf<T, U, NT>), dim3(gx), dim3(kThreads), lds, st, ax,
                     nslices - 1);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.max_split > 0) {
    const unsigned cg = (unsigned)(a.max_split < 4096 ? a.max_split : 4096);
    hipLaunchKernelGGL(k_combine<T>, dim3(cg), dim3(kThreads), 0, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t tiles = (a.max_split + kThreads / 4 - 1) / (kThreads / 4);
    hipLaunchKernelGGL((k_xf_rows<T, NT>), dim3((unsigned)(tiles < 1024 ? tiles : 1024)),
                       dim3(kThreads), lds, st, a);
    e = hipGetLastError();
  }
  return e;
}

template <typename T>
hipError_t launch_xf_nt(const GatherArgs& a, unsigned grid, int nslices, hipStream_t st) {
  switch ((a.xn + 15) / 16) {
    case 1: return launch_xf<T, 1>(a, grid, nslices, st);
    case 2: return launch_xf<T, 2>(a, grid, nslices, st);
    case 3: return launch_xf<T, 3>(a, grid, nslices, st);
    default: return launch_xf<T, 4>(a, grid, nslices, st);
  }
}

}  // namespace

hipError_t launch_gather_transform(const GatherArgs& a0, hipStream_t st) {
  GatherArgs a = a0;
  a.bpw = blocks_per_wg(a);
  const unsigned grid = (unsigned)(a.max_blocks > 0 ? (a.max_blocks + a.bpw - 1) / a.bpw : 1);
  const int esz = a.dtype == SAGA_BF16 ? 2 : 4;
  const int nslices = (int)(a.feat * (int64_t)esz / 128);
  a.xldwt = (int)(a.feat * esz / 16 + 1);
  return a.dtype == SAGA_BF16 ? launch_xf_nt<uint16_t>(a, grid, nslices, st)
                              : launch_xf_nt<float>(a, grid, nslices, st);
}

namespace {

// segment reduction over a contiguous edge tensor: whole rows per lane group
// (the tensor is streamed once, so no slicing for cache reuse)
template <typename T>
hipError_t launch_ident(const GatherArgs& a, int nv, unsigned blocks, hipStream_t st) {
  if (nv > 128) return launch_simple_lpr<T, 8, 1>(a, blocks, (nv + 7) / 8, st);
  if (nv > 64) return launch_simple_lpr<T, 64, 2>(a, blocks, 1, st);
  switch (next_pow2(nv)) {
    case 1: return launch_simple_lpr<T, 1, 1>(a, blocks, 1, st);
    case 2: return launch_simple_lpr<T, 2, 1>(a, blocks, 1, st);
    case 4: return launch_simple_lpr<T, 4, 1>(a, blocks, 1, st);
    case 8: return launch_simple_lpr<T, 8, 1>(a, blocks, 1, st);
    case 16: return launch_simple_lpr<T, 16, 1>(a, blocks, 1, st);
    case 32: return launch_simple_lpr<T, 32, 1>(a, blocks, 1, st);
    default: return launch_simple_lpr<T, 64, 1>(a, blocks, 1, st);
  }
}

template <typename T>
hipError_t launch_select(const GatherArgs& a, int nv, int64_t E, void* msg, int64_t ldm,
                         hipStream_t st) {
  const int64_t total = E * nv;
  const unsigned grid = (unsigned)std::min<int64_t>((total + kThreads - 1) / kThreads, 1 << 16);
  const int64_t ld16 = a.ld_src * (int64_t)sizeof(T) / 16, ldm16 = ldm * (int64_t)sizeof(T) / 16;
  const uint4* src = static_cast<const uint4*>(a.src);
  if (a.msg == SAGA_MSG_SRC_NORM)
    hipLaunchKernelGGL((k_index_select<T, true>), dim3(grid), dim3(kThreads), 0, st, a.col_idx, E,
                       nv, src, ld16, a.d_out, static_cast<uint4*>(msg), ldm16, a.counts);
  else
    hipLaunchKernelGGL((k_index_select<T, false>), dim3(grid), dim3(kThreads), 0, st, a.col_idx,
                       E, nv, src, ld16, a.d_out, static_cast<uint4*>(msg), ldm16, a.counts);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_unfused(const GatherArgs& a0, int64_t E, void* msg, int64_t ldm,
                          hipStream_t st) {
  const int esz = a0.dtype == SAGA_BF16 ? 2 : 4;
  const int nv = (int)((a0.feat * (int64_t)esz + 15) / 16);
  hipError_t err = hipSuccess;
  if (E > 0)
    err = a0.dtype == SAGA_BF16 ? launch_select<uint16_t>(a0, nv, E, msg, ldm, st)
                                : launch_select<float>(a0, nv, E, msg, ldm, st);
  if (err != hipSuccess) return err;
  GatherArgs a = a0;
  a.msg = SAGA_MSG_COPY;
  a.identity = 1;
  a.src = msg;
  a.ld_src = ldm;
  a.bpw = 1;
  const unsigned grid = (unsigned)(a.max_blocks > 0 ? a.max_blocks : 1);
  err = a.dtype == SAGA_BF16 ? launch_ident<uint16_t>(a, nv, grid, st)
                             : launch_ident<float>(a, nv, grid, st);
  if (err != hipSuccess) return err;
  if (a.max_split > 0) {
    const unsigned cg = (unsigned)(a.max_split < 4096 ? a.max_split : 4096);
    if (a.dtype == SAGA_BF16)
      hipLaunchKernelGGL(k_combine<uint16_t>, dim3(cg), dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(k_combine<float>, dim3(cg), dim3(kThreads), 0, st, a);
    err = hipGetLastError();
  }
  return err;
}

hipError_t launch_fold_attention(const float* w, int64_t K, int64_t F, int heads, const float* al,
                                 const float* ar, float* w_ext, int64_t ld_ext, hipStream_t st) {
  const int64_t n = K * (F + 2 * heads);
  const unsigned grid = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(k_fold_attention, dim3(grid), dim3(256), 0, st, w, K, F, heads, al, ar, w_ext,
                     ld_ext);
  return hipGetLastError();
}

}  // namespace saga
