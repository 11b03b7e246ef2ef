// LSTM Gather of GraphSAGE (Table I, GraphSAGE row; Sec. 3.2, Gather
// paragraph): the in-edges of a destination, in CSR order, are the input
// sequence of an LSTM that starts from h = c = 0; the aggregate is its last
// hidden state.  The paper singles this Gather out as the one that cannot be
// fused: it is a recurrence along each row.
//
// Split of the work:
//   * the input half of every gate pre-activation depends only on the
//     source vertex, so it is one dense product over all vertices,
//     P = X W_ih + b_ih + b_hh (the caller's ApplyVertex GEMM), not a
//     product per edge;
//   * what is left per edge is the recurrent step
//       z = P[u_t] + h W_hh;  i, f, o = sigmoid, g = tanh (blocks i|f|g|o);
//       c = f c + i g;  h = o tanh(c)
//     which this kernel runs.
//
// Schedule.  Instead of one launch per distinct degree (the degree traversal
// the paper measured), a persistent grid pulls rows from a work queue in
// degree-sorted order (the plan's perm: longest rows first, so the longest
// recurrence starts at once while the short rows fill the other CUs).  One
// workgroup of 1024 threads runs one row at a time:
//   * W_hh lives in registers: thread t owns gate column j = t / SPLIT and
//     the KPT = H / SPLIT recurrent weights W_hh[k][j] of its k range;
//   * h is in LDS; each step, thread t forms its partial dot product, the
//     SPLIT partials are summed by cross-lane shuffles, the gate is
//     activated into LDS, and H threads update (c, h);
//   * the P rows of the next PF steps are loaded straight into an LDS ring
//     (global_load_lds_dwordx4) by the first waves, so the recurrence never
//     waits on memory; the neighbour ids come in chunks through LDS.
#include <algorithm>

#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kLstmThreads = 1024;
constexpr int kPF = 12;      // P rows in flight ahead of the recurrence
constexpr int kUch = 1024;   // neighbour ids per LDS chunk
constexpr int kLone = 2048;  // the longest rows are handed out one by one
constexpr int kBatch = 8;    // then batches of rows per ticket

typedef __attribute__((address_space(3))) void* lds_ptr;

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt out of range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// wait until at most n (0 <= n < kPF) of this wave's loads are pending
__device__ __forceinline__ void wait_vm_le(int n) {
  switch (n) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<1>(); break;
    case 2: wait_vm<2>(); break;
    case 3: wait_vm<3>(); break;
    case 4: wait_vm<4>(); break;
    case 5: wait_vm<5>(); break;
    case 6: wait_vm<6>(); break;
    case 7: wait_vm<7>(); break;
    case 8: wait_vm<8>(); break;
    case 9: wait_vm<9>(); break;
    case 10: wait_vm<10>(); break;
    default: wait_vm<11>(); break;
  }
  static_assert(kPF == 12, "wait_vm_le covers 0 .. kPF - 1");
}

// A workgroup barrier that orders LDS only: the direct-to-LDS loads in
// flight are waited for explicitly by the waves that issued them.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__global__ void k_lstm_zero(int32_t* q) {
  if (threadIdx.x == 0) q[0] = 0;
}

template <int H>
struct LstmCfg {
  static constexpr int G = 4 * H;                    // gate columns
  static constexpr int SPLIT = kLstmThreads / G;     // threads per gate column
  static constexpr int KPT = H / SPLIT;              // recurrent weights per thread
  static constexpr int PV = G / 4;                   // 16-byte pieces of one P row
  static_assert(SPLIT >= 1 && (SPLIT & (SPLIT - 1)) == 0 && KPT % 4 == 0, "shape");
  static_assert(PV % 64 == 0 || PV < 64, "P row = whole waves or one partial wave");
};

template <int H>
__global__ __launch_bounds__(kLstmThreads) void k_lstm_gather(LstmArgs a) {
  typedef LstmCfg<H> C;
  constexpr int G = C::G, SPLIT = C::SPLIT, KPT = C::KPT, PV = C::PV;
  __shared__ __attribute__((aligned(16))) float ring[(kPF + 1) * G];
  __shared__ __attribute__((aligned(16))) float hbuf[H];
  __shared__ float act[G];
  __shared__ int32_t ucache[2][kUch];
  __shared__ int s_item[2];
  if (a.counts[kErrFlags]) return;

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int j = t / SPLIT, q = t % SPLIT;  // gate column, part of the k range
  const int k0 = q * KPT;
  float w[KPT];
#pragma unroll
  for (int k = 0; k < KPT; ++k) w[k] = a.w_hh[(int64_t)(k0 + k) * a.ld_whh + j];
  const bool tanh_gate = j >= 2 * H && j < 3 * H;
  // P row pieces: lane l of wave w (w * 64 + l < PV) loads piece w * 64 + l
  const bool p_loader = wave * 64 < PV;
  const bool p_lane = wave * 64 + lane < PV;

  int par = 0;
  for (;;) {
    // ticket k: the single row k for the kLone longest rows, then batches of
    // kBatch consecutive rows (fewer same-address atomics for the many
    // short rows, while no long row waits behind another)
    if (t == 0) s_item[par] = atomicAdd(a.queue, 1);
    lds_barrier();
    const int ticket = s_item[par];
    par ^= 1;
    const int64_t first = ticket < kLone ? ticket : kLone + (int64_t)(ticket - kLone) * kBatch;
    if (first >= a.num_dst) break;  // uniform: every thread read the same ticket
    const int64_t last = ticket < kLone ? first + 1 : std::min<int64_t>(first + kBatch, a.num_dst);
    for (int64_t item = first; item < last; ++item) {
    const int v = a.perm[item];
    const int64_t beg = a.row_ptr[v];
    const int d = a.row_ptr[v + 1] - a.row_ptr[v];
    float* orow = a.out + (int64_t)v * a.ld_out;
    if (d <= 0) {
      if (t < H) orow[t] = 0.0f;
      continue;
    }
    lds_barrier();  // the previous row of this ticket is done with hbuf / ucache
    // neighbour ids of chunks 0 and 1; h = 0
    for (int i = t; i < 2 * kUch; i += kLstmThreads)
      if (i < d) ucache[i / kUch][i % kUch] = a.col_idx[beg + i];
    if (t < H) hbuf[t] = 0.0f;
    float c = 0.0f;
    lds_barrier();
    // P rows of the first kPF steps into ring slots 0 .. kPF-1
    if (p_loader) {
      for (int s = 0; s < kPF; ++s) {
        if (s < d) {
          const int u = ucache[0][s];
          if (p_lane)
            __builtin_amdgcn_global_load_lds(a.gates_x + (int64_t)u * a.ld_gx + (wave * 64 + lane) * 4,
                                             (lds_ptr)(ring + s * G + wave * 256), 16, 0, 0);
        }
      }
    }
    for (int s = 0; s < d; ++s) {
      // this wave's P row of step s has landed (the loads of at most the
      // kPF - 1 later steps may still be pending), then everyone's
      if (p_loader) wait_vm_le(std::min(kPF - 1, d - 1 - s));
      lds_barrier();
      // gate pre-activation z_j = P[u_s][j] + sum_k h[k] W_hh[k][j]
      float dot = 0.0f;
#pragma unroll
      for (int k = 0; k < KPT; k += 4) {
        const float4 hv = *reinterpret_cast<const float4*>(hbuf + k0 + k);
        dot += w[k] * hv.x + w[k + 1] * hv.y + w[k + 2] * hv.z + w[k + 3] * hv.w;
      }
#pragma unroll
      for (int off = 1; off < SPLIT; off <<= 1) dot += __shfl_xor(dot, off, 64);
      if (q == 0) {
        const float z = dot + ring[(s % (kPF + 1)) * G + j];
        act[j] = tanh_gate ? tanhf(z) : sigmoidf_(z);
      }
      // the P row of step s + kPF (its slot was last read at step s - 1)
      const int sn = s + kPF;
      if (p_loader && sn < d) {
        const int u = ucache[(sn / kUch) & 1][sn % kUch];
        if (p_lane)
          __builtin_amdgcn_global_load_lds(a.gates_x + (int64_t)u * a.ld_gx + (wave * 64 + lane) * 4,
                                           (lds_ptr)(ring + (sn % (kPF + 1)) * G + wave * 256), 16, 0,
                                           0);
      }
      lds_barrier();
      if (t < H) {
        const float gi = act[t], gf = act[H + t], gg = act[2 * H + t], go = act[3 * H + t];
        c = gf * c + gi * gg;
        const float hn = go * tanhf(c);
        hbuf[t] = hn;
        if (s == d - 1) orow[t] = hn;
      }
      // entering chunk cc: chunk cc + 1 replaces chunk cc - 1, whose ids were
      // last used for the loads of step cc * kUch - 1
      if ((s + 1) % kUch == 0) {
        const int cc = (s + 1) / kUch;
        lds_barrier();
        for (int i = t; i < kUch; i += kLstmThreads) {
          const int64_t e = (int64_t)(cc + 1) * kUch + i;
          if (e < d) ucache[(cc + 1) & 1][i] = a.col_idx[beg + e];
        }
      }
    }
    }  // rows of the ticket
  }
}

template <int H>
hipError_t launch_h(const LstmArgs& a, hipStream_t st) {
  // one resident workgroup per slot: CUs x workgroups that fit per CU
  static int grid = [] {
    int dev = 0, cus = 256, per = 1;
    if (hipGetDevice(&dev) == hipSuccess)
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, k_lstm_gather<H>, kLstmThreads, 0) !=
            hipSuccess || per < 1)
      per = 1;
    return (cus > 0 ? cus : 256) * per;
  }();
  hipLaunchKernelGGL(k_lstm_zero, dim3(1), dim3(64), 0, st, a.queue);
  hipLaunchKernelGGL((k_lstm_gather<H>), dim3(grid), dim3(kLstmThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lstm_gather(const LstmArgs& a, hipStream_t st) {
  if (a.num_dst == 0) return hipSuccess;
  switch (a.hidden) {
    case 32: return launch_h<32>(a, st);
    case 64: return launch_h<64>(a, st);
    case 128: return launch_h<128>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace saga
