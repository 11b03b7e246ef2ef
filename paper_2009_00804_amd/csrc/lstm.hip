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
// workgroup of 4H threads runs one row at a time; the longest row's d
// sequential steps bound the time, so a step is kept as short as the vector
// ALU allows (4H x H multiply-adds per step):
//   * thread t serves hidden unit i = t / 4 and the quarter q = t % 4 of the
//     recurrent sum: it keeps the H/4 x 4 weights W_hh[k][gate * H + i]
//     (k in its quarter, the four gates of unit i) in registers, so every h
//     value it reads from LDS feeds four multiply-adds;
//   * the unit's four lanes (a quad) reduce-scatter their partial sums with
//     DPP quad permutations, so lane q holds gate q's pre-activation and
//     applies that gate's activation alone; the four activations are then
//     broadcast within the quad, every lane updates its copy of (c, h), and
//     lane 0 writes h to a double-buffered LDS vector -- one workgroup
//     barrier per step;
//   * the P rows of the next PF steps are loaded straight into an LDS ring
//     (global_load_lds_dwordx4) by the first waves, so the recurrence never
//     waits on memory; the neighbour ids come in chunks through LDS.
// The same kernel takes a range of perm positions, so a caller can also run
// the degree traversal (one launch per run of equal degrees) for comparison.
#include <algorithm>

#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kSplit = 4;    // threads per hidden unit (quarters of the recurrent sum)
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

// Gate functions with the hardware reciprocal (about 1 ulp) instead of a
// correctly rounded division, which costs ten instructions:
// sigmoid(x) = 1 / (1 + exp(-x)); tanh(x) = 1 - 2 / (exp(2x) + 1) (saturates
// to +-1 for large |x|; near 0 its absolute error is at the float32 rounding
// level).
__device__ __forceinline__ float sigmoid_fast(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}
__device__ __forceinline__ float tanh_fast(float x) {
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(__expf(2.0f * x) + 1.0f);
}

// Quad (four-lane) exchanges through DPP quad permutations; a generic
// shuffle would go through the LDS crossbar (ds_bpermute) and add its
// latency to every step.  quad_xor<M>: the value of lane ^ M; quad_bcast<K>:
// the value of lane K of the quad.
template <int M>
__device__ __forceinline__ float quad_xor(float x) {
  static_assert(M == 1 || M == 2, "quad lane mask");
  constexpr int ctrl = M == 1 ? 0xB1 : 0x4E;  // quad_perm [1,0,3,2] / [2,3,0,1]
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), ctrl, 0xF, 0xF, false));
}
template <int K>
__device__ __forceinline__ float quad_bcast(float x) {
  static_assert(K >= 0 && K < 4, "quad lane");
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), K * 0x55, 0xF, 0xF, false));
}

__global__ void k_lstm_zero(int32_t* q) {
  if (threadIdx.x == 0) q[0] = 0;
}

template <int H>
struct LstmCfg {
  static constexpr int G = 4 * H;                // gate columns
  static constexpr int THREADS = kSplit * H;     // 128, 256 or 512
  static constexpr int KPT = H / kSplit;         // recurrent k per thread
  static constexpr int PV = G / 4;               // 16-byte pieces of one P row
  static_assert(KPT % 4 == 0, "shape");
  static_assert(PV % 64 == 0 || PV < 64, "P row = whole waves or one partial wave");
  static_assert(PV <= THREADS, "P row loaders");
};

template <int H>
__global__ __launch_bounds__(LstmCfg<H>::THREADS) void k_lstm_gather(LstmArgs a) {
  typedef LstmCfg<H> C;
  constexpr int G = C::G, KPT = C::KPT, PV = C::PV, NT = C::THREADS;
  __shared__ __attribute__((aligned(16))) float ring[(kPF + 1) * G];
  __shared__ __attribute__((aligned(16))) float hbuf[2][H];
  __shared__ int32_t ucache[2][kUch];
  __shared__ int s_item[2];
  if (a.counts[kErrFlags]) return;

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int i = t / kSplit, q = t % kSplit;  // hidden unit, quarter of the k range
  const int k0 = q * KPT;
  float w[4][KPT];
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int k = 0; k < KPT; ++k) w[g][k] = a.w_hh[(int64_t)(k0 + k) * a.ld_whh + g * H + i];
  // P row pieces: lane l of wave w (w * 64 + l < PV) loads piece w * 64 + l
  const bool p_loader = wave * 64 < PV;
  const bool p_lane = wave * 64 + lane < PV;
  const int64_t npos = (int64_t)a.perm_end - a.perm_begin;
  const uint32_t ring_base = (uint32_t)reinterpret_cast<uintptr_t>((lds_ptr)ring);

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
    if (first >= npos) break;  // uniform: every thread read the same ticket
    const int64_t last = ticket < kLone ? first + 1 : std::min<int64_t>(first + kBatch, npos);
    for (int64_t item = first; item < last; ++item) {
      const int v = a.perm[a.perm_begin + item];
      const int64_t beg = a.row_ptr[v];
      const int d = a.row_ptr[v + 1] - a.row_ptr[v];
      float* orow = a.out + (int64_t)v * a.ld_out;
      if (d <= 0) {
        if (t < H) orow[t] = 0.0f;
        continue;
      }
      // the previous row's output stores have drained, so the vmcnt waits
      // below count this row's ring loads only; the previous row is done
      // with hbuf and ucache
      wait_vm<0>();
      lds_barrier();
      // neighbour ids of chunks 0 and 1; h = 0
      for (int j = t; j < 2 * kUch; j += NT)
        if (j < d) ucache[j / kUch][j % kUch] = a.col_idx[beg + j];
      if (t < H) hbuf[0][t] = 0.0f;
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
        // kPF - 1 later steps may still be pending), then everyone's; h of
        // step s - 1 is in hbuf[s & 1]
        if (p_loader) wait_vm_le(std::min(kPF - 1, d - 1 - s));
        lds_barrier();
        // this lane's gate-q entry of the step's P row, read with an inline
        // ds_read_b32 and waited for after the recurrent sum: read as plain
        // C++, the compiler would first wait for every direct-to-LDS load in
        // flight (they may write the ring), stalling each step on the newest
        // prefetch.  The slot has landed: its loader waves waited for it
        // before the barrier.
        float pq;
        asm volatile("ds_read_b32 %0, %1"
                     : "=v"(pq)
                     : "v"(ring_base + (uint32_t)(((s % (kPF + 1)) * G + q * H + i) * 4))
                     : "memory");
        // this thread's quarter of h, all of it read before the first
        // multiply-add (one LDS wait per step)
        const float* hb = hbuf[s & 1];
        float hk[KPT];
#pragma unroll
        for (int k = 0; k < KPT; k += 4) {
          const float4 hv = *reinterpret_cast<const float4*>(hb + k0 + k);
          hk[k] = hv.x;
          hk[k + 1] = hv.y;
          hk[k + 2] = hv.z;
          hk[k + 3] = hv.w;
        }
        __builtin_amdgcn_sched_barrier(0);  // keep every read ahead of the multiply-adds
        float z0 = 0.0f, z1 = 0.0f, z2 = 0.0f, z3 = 0.0f;
#pragma unroll
        for (int k = 0; k < KPT; ++k) {  // four independent chains
          z0 = fmaf(w[0][k], hk[k], z0);
          z1 = fmaf(w[1][k], hk[k], z1);
          z2 = fmaf(w[2][k], hk[k], z2);
          z3 = fmaf(w[3][k], hk[k], z3);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(pq) : : "memory");
        // reduce-scatter over the quad: lane q ends with the full sum of gate
        // q (lane ^ 2 exchanges gate pairs, lane ^ 1 single gates)
        const bool hi = q & 2, odd = q & 1;
        float k0 = hi ? z2 : z0, k1 = hi ? z3 : z1;
        k0 += quad_xor<2>(hi ? z0 : z2);
        k1 += quad_xor<2>(hi ? z1 : z3);
        const float zq = (odd ? k1 : k0) + quad_xor<1>(odd ? k0 : k1) + pq;
        // gate q's activation: tanh for g (q == 2, as 2 sigmoid(2x) - 1),
        // sigmoid for i, f, o; then all four to every lane of the quad
        const float sg = sigmoid_fast(q == 2 ? 2.0f * zq : zq);
        const float aq = q == 2 ? 2.0f * sg - 1.0f : sg;
        const float gi = quad_bcast<0>(aq), gf = quad_bcast<1>(aq), gg = quad_bcast<2>(aq),
                    go = quad_bcast<3>(aq);
        c = gf * c + gi * gg;
        const float hn = go * tanh_fast(c);
        if (q == 0) {
          hbuf[(s + 1) & 1][i] = hn;
          if (s == d - 1) orow[i] = hn;
        }
        // the P row of step s + kPF goes to the slot step s - 1 used (read
        // before this step's barrier)
        const int sn = s + kPF;
        if (p_loader && sn < d) {
          const int u = ucache[(sn / kUch) & 1][sn % kUch];
          if (p_lane)
            __builtin_amdgcn_global_load_lds(a.gates_x + (int64_t)u * a.ld_gx + (wave * 64 + lane) * 4,
                                             (lds_ptr)(ring + (sn % (kPF + 1)) * G + wave * 256), 16,
                                             0, 0);
        }
        // entering chunk cc: chunk cc + 1 replaces chunk cc - 1, whose ids
        // were last read for the load of step cc * kUch - 1 (issued kPF
        // steps, and barriers, ago)
        if ((s + 1) % kUch == 0) {
          const int cc = (s + 1) / kUch;
          for (int j = t; j < kUch; j += NT) {
            const int64_t e = (int64_t)(cc + 1) * kUch + j;
            if (e < d) ucache[(cc + 1) & 1][j] = a.col_idx[beg + e];
          }
        }
      }
    }  // rows of the ticket
  }
}

template <int H>
hipError_t launch_h(const LstmArgs& a, hipStream_t st) {
  // one workgroup per CU: the longest row's step time is what bounds the
  // call, so it does not share its CU's vector ALUs with a second row
  static int grid = [] {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
      (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    return cus > 0 ? cus : 256;
  }();
  const int64_t n = (int64_t)a.perm_end - a.perm_begin;
  const unsigned g = (unsigned)std::min<int64_t>(grid, n);
  hipLaunchKernelGGL(k_lstm_zero, dim3(1), dim3(64), 0, st, a.queue);
  hipLaunchKernelGGL((k_lstm_gather<H>), dim3(g), dim3(LstmCfg<H>::THREADS), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lstm_gather(const LstmArgs& a, hipStream_t st) {
  if (a.perm_end <= a.perm_begin) return hipSuccess;
  switch (a.hidden) {
    case 32: return launch_h<32>(a, st);
    case 64: return launch_h<64>(a, st);
    case 128: return launch_h<128>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace saga
