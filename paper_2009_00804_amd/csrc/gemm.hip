// ApplyVertex: the dense per-vertex transform (Sec. 3.2 "ApplyVertex" of
// the paper: all vertices batched into one GEMM, Table III) on the CDNA4
// matrix cores, with the layer's epilogue fused (degree row scaling, bias,
// activation, the two-operand concat form [a | a2][w ; w2], and the GRU
// gate math of GGNN's ApplyVertex, Fig. 2).
//
// Tiling: a workgroup of 4 waves owns BM = 64 MT rows and BN = 16 NT
// columns; wave w computes rows [16 MT w, 16 MT (w + 1)) of the tile as
// MT x NT blocks of 16 x 16 with
//   float32 : v_mfma_f32_16x16x4f32   (4 k per instruction)
//   bfloat16: v_mfma_f32_16x16x32_bf16 (32 k per instruction)
//
// Data path.  K is cut into chunks of 128 bytes per row (32 float32 or 64
// bfloat16 values).  For every chunk the BM rows of A and the BN rows of the
// packed weights Wt (W transposed, zero-padded to whole tiles, built in the
// workspace by k_pack_wt) go straight from global memory into one stage of
// an S-stage LDS ring with direct-to-LDS loads (global_load_lds_dwordx4).
// Nothing is staged through registers, so the loads of later stages never
// wait behind one another and S - 1 chunks stay in flight while one is
// multiplied.  Inside a 128-byte row the eight 16-byte pieces are XOR
// swizzled (piece p of row r at slot 8 r + (p ^ ((r >> 1) & 7))), so that a
// fragment read -- 16 rows at one k offset -- touches every LDS bank once.
// A lane's 16-byte fragment holds EPL consecutive k of one row; A and Wt
// use the same k order, so the products are exact sums over k.
//
// The chunk holding the end of K is loaded first, through registers, with
// zeros past column K and past row M; every later chunk is a whole 128-byte
// row segment and needs no masking in k.
#include <algorithm>
#include <type_traits>
#include <cstdlib>
#include <cstring>

#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kThreads = 256;

typedef __attribute__((address_space(3))) void* lds_ptr;

template <typename T> struct Mma;

template <> struct Mma<float> {
  static constexpr int EPL = 4;     // elements per 16-byte fragment
  static constexpr int KC = 32;     // k per 128-byte chunk
  typedef f32x4 Frag;
  __device__ __forceinline__ static float to_f(float x) { return x; }
  __device__ __forceinline__ static float from_f(float x) { return x; }
};

template <> struct Mma<uint16_t> {
  static constexpr int EPL = 8;
  static constexpr int KC = 64;
  typedef bf16x8 Frag;
  __device__ __forceinline__ static float to_f(uint16_t x) { return bf16_to_f32(x); }
  __device__ __forceinline__ static uint16_t from_f(float x) { return f32_to_bf16(x); }
};

__device__ __forceinline__ int swz(int r, int p) { return r * 8 + (p ^ ((r >> 1) & 7)); }

// s_waitcnt vmcnt(N) (gfx9 encoding; expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt out of range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for the LDS ring.  A plain __syncthreads() would also
// wait for every direct-to-LDS load in flight (its release fence covers LDS
// writes, and those loads write LDS), which would drain the ring at every
// chunk.  Here the caller has already waited for the stage it needs; the
// barrier only orders this wave's own LDS reads and writes.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <typename T, int MT, int NT, int S>
struct Ring {
  static constexpr int BM = 64 * MT, BN = 16 * NT;
  static constexpr int A_SLOTS = BM * 8, B_SLOTS = BN * 8;  // 16-byte slots
  static constexpr int STAGE = A_SLOTS + B_SLOTS;
  static constexpr int RING_SLOTS = S * STAGE;
  static constexpr int THREADS = kThreads;
  static constexpr int LA = A_SLOTS / kThreads;              // loads per thread per stage
  static constexpr int LB = (B_SLOTS + kThreads - 1) / kThreads;
  // fewest loads any wave issues per stage (waves past the end of a partial
  // B row skip the last one); waiting on this count is exact or conservative
  static constexpr int LMIN = LA + B_SLOTS / kThreads;
  static_assert(A_SLOTS % kThreads == 0, "A tile must be whole wave loads");
  static_assert(B_SLOTS % 64 == 0, "B tile must be whole wave loads");
  static_assert((S - 2) * LMIN < 64, "vmcnt range");
  static_assert(S >= 2, "at least two stages");
  static constexpr size_t LDS_BYTES = (size_t)S * STAGE * 16;

  // direct-to-LDS loads of chunk k0 of rows [row0, row0 + BM) of A (rows
  // >= M skipped) and rows [n0, n0 + BN) of Wt into one stage
  __device__ __forceinline__ static void issue_a(const T* __restrict__ A, int64_t lda, int64_t M,
                                                 int64_t row0, int64_t k0, uint4* st) {
    constexpr int EPL = Mma<T>::EPL;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < LA; ++j) {
      const int s0 = j * kThreads + wave * 64;
      const int s = s0 + lane, r = s >> 3, p = (s & 7) ^ ((r >> 1) & 7);
      if (row0 + r < M)
        __builtin_amdgcn_global_load_lds(A + (row0 + r) * lda + k0 + p * EPL, (lds_ptr)(st + s0), 16, 0, 0);
    }
  }
  __device__ __forceinline__ static void issue_b(const T* __restrict__ Wt, int64_t kp, int64_t n0,
                                                 int64_t k0, uint4* st) {
    constexpr int EPL = Mma<T>::EPL;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < LB; ++j) {
      const int s0 = j * kThreads + wave * 64;
      if (s0 < B_SLOTS) {
        const int s = s0 + lane, n = s >> 3, p = (s & 7) ^ ((n >> 1) & 7);
        __builtin_amdgcn_global_load_lds(Wt + (n0 + n) * kp + k0 + p * EPL,
                                         (lds_ptr)(st + A_SLOTS + s0), 16, 0, 0);
      }
    }
  }

  // vmcnt wait that leaves only the loads of the next `later` stages pending;
  // `tail` says the last of them is the K-tail stage, which issues only its
  // B loads (its A part was loaded into registers before every other load)
  static constexpr int LBMIN = B_SLOTS / kThreads;
  __device__ __forceinline__ static void wait_stages(int later, bool tail) {
    if constexpr (S >= 4) {
      if (later >= 2) {
        if (tail) wait_vm<LMIN + LBMIN>(); else wait_vm<2 * LMIN>();
        return;
      }
    }
    if constexpr (S >= 3) {
      if (later == 1) {
        if (tail) wait_vm<LBMIN>(); else wait_vm<LMIN>();
        return;
      }
    }
    wait_vm<0>();
  }

  // The A tail chunk through registers.  A piece that starts below K is
  // loaded whole (it ends within the row's ld, which is a multiple of 16
  // bytes); the values at columns >= K, and whole pieces past row M or
  // column K, are zeroed when the piece is written to LDS.  The loads are
  // unconditional, so nothing has to wait for them before the stage opens.
  struct Tail {
    uint4 v[LA];
    int nv[LA];  // valid elements of each piece (0 .. EPL)
    __device__ __forceinline__ void load(const T* __restrict__ A, int64_t lda, int64_t M, int64_t K,
                                         int64_t row0, int64_t k0) {
      constexpr int EPL = Mma<T>::EPL;
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
      for (int j = 0; j < LA; ++j) {
        const int s = j * kThreads + wave * 64 + lane, r = s >> 3, p = (s & 7) ^ ((r >> 1) & 7);
        const int64_t row = row0 + r, k = k0 + p * EPL;
        const int64_t left = K - k;
        nv[j] = row < M ? (int)(left <= 0 ? 0 : left >= EPL ? EPL : left) : 0;
        // pieces with nothing valid read an in-range piece instead (no branch)
        const int64_t rr = row < M ? row : M - 1;
        const int64_t kk = left > 0 ? k : (K - 1) / EPL * EPL;
        v[j] = *reinterpret_cast<const uint4*>(A + rr * lda + kk);
      }
    }
    __device__ __forceinline__ void store(uint4* st) const {
      constexpr int EPL = Mma<T>::EPL;
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
      for (int j = 0; j < LA; ++j) {
        uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          if constexpr (EPL == 4) {
            if (d >= nv[j]) w[d] = 0;
          } else {  // two bfloat16 per word
            if (2 * d >= nv[j]) w[d] = 0;
            else if (2 * d + 1 >= nv[j]) w[d] &= 0xffffu;
          }
        }
        st[j * kThreads + wave * 64 + lane] = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
  };

  // acc += (one chunk of A rows of this wave) x (chunk of Wt).  All
  // fragments of the chunk are read before the first MFMA, so the reads of
  // the second k-step complete under the MFMAs of the first.
  __device__ __forceinline__ static void compute(const uint4* st, f32x4 (&acc)[MT][NT]) {
    typedef typename Mma<T>::Frag Frag;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const uint4* As = st;
    const uint4* Bs = st + A_SLOTS;
    Frag a[2][MT], b[2][NT];
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // two k-steps of 64 bytes
      const int p = h * 4 + lg;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const uint4 v = As[swz(wave * MT * 16 + mt * 16 + lr, p)];
        __builtin_memcpy(&a[h][mt], &v, 16);
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const uint4 v = Bs[swz(nt * 16 + lr, p)];
        __builtin_memcpy(&b[h][nt], &v, 16);
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[h][mt][c], b[h][nt][c], acc[mt][nt], 0, 0, 0);
      } else {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[h][mt], b[h][nt], acc[mt][nt], 0, 0, 0);
      }
    }
  }

  // acc += A[row0 .. row0 + BM) x W[:, n0 .. n0 + BN), W given packed as Wt
  // (ld kp, zero-padded).  Stage j holds chunk j.  Chunks 0 .. nch-2 are
  // whole and loaded direct-to-LDS.  The A part of the last one (the K tail)
  // is loaded into registers before anything else and written to LDS just
  // before the barrier that opens its stage; its B part is loaded like the
  // others.  Loads complete in issue order, so waiting until at most the
  // loads of the stages issued after stage i are pending means stage i has
  // landed; the counts used are the fewest any wave issues.
  __device__ __forceinline__ static void phase(const T* __restrict__ A, int64_t lda, int64_t M,
                                               int64_t K, const T* __restrict__ Wt, int64_t kp,
                                               int64_t row0, int64_t n0, uint4* ring,
                                               f32x4 (&acc)[MT][NT]) {
    constexpr int KC = Mma<T>::KC;
    const int nch = (int)((K + KC - 1) / KC);
    const int last = nch - 1;
    Tail tail;
    tail.load(A, lda, M, K, row0, (int64_t)last * KC);
    auto issue = [&](int j) {
      uint4* st = ring + (j % S) * STAGE;
      if (j < last) issue_a(A, lda, M, row0, (int64_t)j * KC, st);
      issue_b(Wt, kp, n0, (int64_t)j * KC, st);
    };
    for (int j = 0; j < S - 1 && j < nch; ++j) issue(j);
    for (int i = 0; i < nch; ++i) {
      const int ahead = last - i;
      const int later = ahead < S - 2 ? ahead : S - 2;
      wait_stages(later, later > 0 && ahead <= S - 2);  // this wave's loads of stage i landed
      if (i == last) tail.store(ring + (i % S) * STAGE);
      ring_barrier();  // ... and every wave's; stage i - 1 is free again
      if (i + S - 1 < nch) issue(i + S - 1);
      compute(ring + (i % S) * STAGE, acc);
    }
    ring_barrier();  // the ring may be refilled by a following phase
  }
};

// Second data path: A straight from global memory into registers, only
// the packed weights through the LDS ring.  Each wave owns its A rows, so
// A needs no sharing through LDS; the ring then holds only the BN x 128-byte
// weight chunks (16 KB per stage for BN = 128), which leaves LDS room for
// more resident workgroups.  A chunk's A and Wt loads are issued together,
// S - 1 chunks ahead, so one vmcnt wait covers both.
template <typename T, int MT, int NT, int S, int NW = 4>
struct RegA {
  typedef typename Mma<T>::Frag Frag;
  static constexpr int THREADS = 64 * NW;  // NW waves, each 16 MT rows
  static constexpr int BM = 16 * MT * NW, BN = 16 * NT;
  static constexpr int B_SLOTS = BN * 8;
  static constexpr int STAGE = B_SLOTS;
  static constexpr int RING_SLOTS = S * STAGE;
  static constexpr int LA = 2 * MT;  // 16-byte A loads per lane per chunk
  static constexpr int LB = (B_SLOTS + THREADS - 1) / THREADS;
  static constexpr int LMIN = LA + B_SLOTS / THREADS;
  static_assert(B_SLOTS % 64 == 0, "B tile must be whole wave loads");
  static_assert(S >= 2 && (S - 2) * LMIN < 64, "vmcnt range");
  static constexpr size_t LDS_BYTES = (size_t)RING_SLOTS * 16;

  // element offsets of this lane's A rows r0 + 16 mt + lane % 16.  Rows >=
  // M read row M - 1 (their results are never stored).  With a row map, row
  // q is row arow[q] of A; a negative entry reads row 0 (the caller writes
  // zeros for it).
  __device__ __forceinline__ static void row_offsets(const int32_t* __restrict__ arow, int64_t lda,
                                                     int64_t M, int64_t r0, int64_t (&off)[MT]) {
    const int lr = threadIdx.x & 15;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int64_t row = r0 + mt * 16 + lr;
      int64_t rr = row < M ? row : M - 1;
      if (arow) {
        const int32_t s = arow[rr];
        rr = s >= 0 ? s : 0;
      }
      off[mt] = rr * lda;
    }
  }

  // fragment (h, mt) of chunk k0: the lane's row mt, columns
  // k0 + (4 h + lane / 16) EPL ..  A piece that starts at or past K reads
  // the last piece of the row instead and is zeroed by mask() before use.  A
  // piece that starts below K ends within the row's ld (a multiple of 16
  // bytes).
  __device__ __forceinline__ static void load_a(const T* __restrict__ A,
                                                const int64_t (&off)[MT], int64_t K, int64_t k0,
                                                Frag (&a)[2][MT]) {
    constexpr int EPL = Mma<T>::EPL;
    const int lane = threadIdx.x & 63, lg = lane >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int64_t k = k0 + (h * 4 + lg) * EPL;
        const int64_t kk = k < K ? k : (K - 1) / EPL * EPL;
        const uint4 v = *reinterpret_cast<const uint4*>(A + off[mt] + kk);
        __builtin_memcpy(&a[h][mt], &v, 16);
      }
  }
  // zero the values at columns >= K (the tail chunk)
  __device__ __forceinline__ static void mask(int64_t K, int64_t k0, Frag (&a)[2][MT]) {
    constexpr int EPL = Mma<T>::EPL;
    const int lg = (threadIdx.x & 63) >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t left = K - (k0 + (h * 4 + lg) * EPL);
      const int nv = left <= 0 ? 0 : left >= EPL ? EPL : (int)left;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        uint32_t w[4];
        __builtin_memcpy(w, &a[h][mt], 16);
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          if constexpr (EPL == 4) {
            if (d >= nv) w[d] = 0;
          } else {
            if (2 * d >= nv) w[d] = 0;
            else if (2 * d + 1 >= nv) w[d] &= 0xffffu;
          }
        }
        __builtin_memcpy(&a[h][mt], w, 16);
      }
    }
  }
  __device__ __forceinline__ static void issue_b(const T* __restrict__ Wt, int64_t kp, int64_t n0,
                                                 int64_t k0, uint4* st) {
    constexpr int EPL = Mma<T>::EPL;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < LB; ++j) {
      const int s0 = j * THREADS + wave * 64;
      if (s0 < B_SLOTS) {
        const int s = s0 + lane, n = s >> 3, p = (s & 7) ^ ((n >> 1) & 7);
        __builtin_amdgcn_global_load_lds(Wt + (n0 + n) * kp + k0 + p * EPL, (lds_ptr)(st + s0), 16, 0, 0);
      }
    }
  }
  __device__ __forceinline__ static void wait_stages(int later) {
    if constexpr (S >= 4) {
      if (later >= 2) { wait_vm<2 * LMIN>(); return; }
    }
    if constexpr (S >= 3) {
      if (later == 1) { wait_vm<LMIN>(); return; }
    }
    wait_vm<0>();
  }
  __device__ __forceinline__ static void compute(const uint4* Bs, const Frag (&a)[2][MT],
                                                 f32x4 (&acc)[MT][NT]) {
    const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
    Frag b[2][NT];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const uint4 v = Bs[swz(nt * 16 + lr, h * 4 + lg)];
        __builtin_memcpy(&b[h][nt], &v, 16);
      }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[h][mt][c], b[h][nt][c], acc[mt][nt], 0, 0, 0);
      } else {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[h][mt], b[h][nt], acc[mt][nt], 0, 0, 0);
      }
    }
  }

  struct Ctx {
    const T* A; int64_t K;
    const T* Wt; int64_t kp, n0;
    int64_t off[MT];
    uint4* ring;
    int nch, last;
  };

  // chunk i = i0 + U: uses register slot U and ring stage U
  template <int U>
  __device__ __forceinline__ static void step(const Ctx& c, int i0, Frag (&a)[S][2][MT],
                                              f32x4 (&acc)[MT][NT]) {
    constexpr int KC = Mma<T>::KC;
    constexpr int NU = (U + S - 1) % S;
    const int i = i0 + U;
    if (i >= c.nch) return;
    wait_stages(c.last - i < S - 2 ? c.last - i : S - 2);  // chunk i's loads landed
    ring_barrier();  // every wave's; stage i - 1 is free again
    if (i + S - 1 < c.nch) {
      load_a(c.A, c.off, c.K, (int64_t)(i + S - 1) * KC, a[NU]);
      issue_b(c.Wt, c.kp, c.n0, (int64_t)(i + S - 1) * KC, c.ring + NU * STAGE);
    }
    if (i == c.last) mask(c.K, (int64_t)i * KC, a[U]);
    compute(c.ring + U * STAGE, a[U], acc);
  }

  // acc += A[tile0 .. tile0 + BM) x W[:, n0 .. n0 + BN); chunk i uses
  // register slot i % S and ring stage i % S (the loop is unrolled by S so
  // both are compile-time)
  __device__ __forceinline__ static void phase(const T* __restrict__ A, int64_t lda, int64_t M,
                                               int64_t K, const T* __restrict__ Wt, int64_t kp,
                                               int64_t tile0, int64_t n0, uint4* ring,
                                               f32x4 (&acc)[MT][NT],
                                               const int32_t* __restrict__ arow = nullptr) {
    static_assert(S <= 4, "unrolled for at most four stages");
    constexpr int KC = Mma<T>::KC;
    Ctx c;
    c.A = A; c.K = K; c.Wt = Wt; c.kp = kp; c.n0 = n0;
    row_offsets(arow, lda, M, tile0 + (threadIdx.x >> 6) * MT * 16, c.off);
    c.ring = ring;
    c.nch = (int)((K + KC - 1) / KC);
    c.last = c.nch - 1;
    Frag a[S][2][MT];
#pragma unroll
    for (int j = 0; j < S - 1; ++j)
      if (j < c.nch) {
        load_a(A, c.off, K, (int64_t)j * KC, a[j]);
        issue_b(Wt, kp, n0, (int64_t)j * KC, ring + j * STAGE);
      }
    for (int i0 = 0; i0 < c.nch; i0 += S) {
      step<0>(c, i0, a, acc);
      step<1>(c, i0, a, acc);
      if constexpr (S > 2) step<2>(c, i0, a, acc);
      if constexpr (S > 3) step<3>(c, i0, a, acc);
    }
    ring_barrier();  // the ring may be refilled by a following phase
  }
};

// Wt[n][k] = W[k][n] for n < N, k < K, else 0; Wt is Np x Kp with ld Kp
template <typename T>
__global__ __launch_bounds__(kThreads) void k_pack_wt(const T* __restrict__ W, int64_t ldw,
                                                      int64_t K, int64_t N, T* __restrict__ Wt,
                                                      int64_t Kp, int64_t Np) {
  const int64_t total = Np * Kp;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t n = i / Kp, k = i - n * Kp;
    Wt[i] = (n < N && k < K) ? W[k * ldw + n] : T(0);
  }
}

// ---------------------------------------------------------------------------
// epilogue.  Lane l of a wave holds rows 4 (l / 16) + r (r < 4), column
// l % 16 of each 16 x 16 accumulator tile (mt, nt).
// ---------------------------------------------------------------------------

template <int ACT, int MT, int NT>
__device__ __forceinline__ void act_tile(f32x4 (&acc)[MT][NT]) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[mt][nt][r] = apply_act(ACT, acc[mt][nt][r]);
}

// Row scale, biases and activation applied to the accumulators in place,
// in that order (v = acc * rs + b1 + b2, then act).  Each optional step is
// one uniform branch around the whole tile, and every load happens before
// the first store (the compiler cannot tell the output from the loaded
// arrays, so a load after a store would wait for it).
template <int MT, int NT>
__device__ __forceinline__ void finish_tile(const GemmArgs& g, int64_t row0, int64_t n0,
                                            f32x4 (&acc)[MT][NT]) {
  const int lane = threadIdx.x & 63;
  if (g.row_scale_deg) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = row0 + mt * 16 + 4 * (lane >> 4) + r;
        const float rs = row < g.M ? rsqrt_deg(g.row_scale_deg[row]) : 0.0f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt][r] *= rs;
      }
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float* bias = k == 0 ? g.bias : g.bias2;
    if (!bias) continue;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int64_t c = n0 + nt * 16 + (lane & 15);
      const float b = c < g.N ? bias[c] : 0.0f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[mt][nt][r] += b;
    }
  }
  switch (g.act) {
    case SAGA_ACT_RELU: act_tile<SAGA_ACT_RELU>(acc); break;
    case SAGA_ACT_ELU: act_tile<SAGA_ACT_ELU>(acc); break;
    case SAGA_ACT_SIGMOID: act_tile<SAGA_ACT_SIGMOID>(acc); break;
    case SAGA_ACT_TANH: act_tile<SAGA_ACT_TANH>(acc); break;
    default: break;
  }
}

// output element (row, c) of the finished tile: columns >= split go to out2
template <typename T>
__device__ __forceinline__ void store_elem(const GemmArgs& g, int64_t row, int64_t c, float v) {
  if (g.split > 0 && c >= g.split)
    static_cast<T*>(g.out2)[row * g.ldo2 + (c - g.split)] = Mma<T>::from_f(v);
  else
    static_cast<T*>(g.out)[row * g.ldo + c] = Mma<T>::from_f(v);
}

// element by element, straight from the accumulators
template <typename T, int MT, int NT>
__device__ __forceinline__ void store_direct(const GemmArgs& g, int64_t row0, int64_t n0,
                                             const f32x4 (&acc)[MT][NT]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = row0 + mt * 16 + 4 * (lane >> 4) + r;
      if (row >= g.M) continue;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int64_t c = n0 + nt * 16 + (lane & 15);
        if (c < g.N) store_elem<T>(g, row, c, acc[mt][nt][r]);
      }
    }
}

// bfloat16, 128 columns from column 0, through registers: three lane
// exchanges (partners lr ^ 1 and lr ^ 2 by DPP, lr ^ 4 by swizzle; lr =
// lane % 16 with bits b0..b3, lg = lane / 16) turn the accumulator layout
// (rows 4 lg + r of column 16 t + lr) into whole 16-byte row pieces: the
// lane then holds, for q = 0..3, row 4 lg + 2 b0 + b1 at columns
// 16 (2 q + b2) + 8 b3 .. + 7, and stores each with one 16-byte store
// (element by element where the piece is not whole, as for the staged
// stores).  For callers whose LDS is taken.
__device__ __forceinline__ uint32_t pack_bf2(uint32_t lo, uint32_t hi) {
  return (lo & 0xffffu) | (hi << 16);
}
template <int MT>
__device__ __forceinline__ void store_shuffled(const GemmArgs& g, int64_t row0,
                                               const f32x4 (&acc)[MT][8]) {
  typedef uint16_t T;
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const bool b0 = lr & 1, b1 = (lr >> 1) & 1, b2 = (lr >> 2) & 1, b3 = (lr >> 3) & 1;
  const bool vec = (reinterpret_cast<uintptr_t>(g.out) & 15) == 0 && (g.ldo * 2) % 16 == 0 &&
                   (g.split <= 0 || ((reinterpret_cast<uintptr_t>(g.out2) & 15) == 0 &&
                                     (g.ldo2 * 2) % 16 == 0));
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    uint32_t z[8][2];  // row 4 lg + 2 b0 + b1, columns 16 t + 4 (lr / 4) .. + 3
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      uint32_t x[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) x[r] = Mma<T>::from_f(acc[mt][nt][r]);
      // lanes with b0 = 0 keep rows 0, 1 and those with b0 = 1 rows 2, 3,
      // now for the column pair (lr & ~1, + 1)
      const uint32_t r1 = (uint32_t)__builtin_amdgcn_mov_dpp(
          (int)(b0 ? pack_bf2(x[0], x[1]) : pack_bf2(x[2], x[3])), 0xB1, 0xF, 0xF, true);
      const uint32_t y0 = b0 ? pack_bf2(r1, x[2]) : pack_bf2(x[0], r1);
      const uint32_t y1 = b0 ? pack_bf2(r1 >> 16, x[3]) : pack_bf2(x[1], r1 >> 16);
      // lanes with b1 = 0 keep the first of the two rows, b1 = 1 the second,
      // now for four columns from lr & ~3
      const uint32_t r2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)(b1 ? y0 : y1), 0x4E, 0xF, 0xF, true);
      z[nt][0] = b1 ? r2 : y0;
      z[nt][1] = b1 ? y1 : r2;
    }
    const int64_t row = row0 + mt * 16 + 4 * lg + 2 * b0 + b1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // lanes with b2 = 0 keep tile 2 q and those with b2 = 1 tile 2 q + 1,
      // now for eight columns from 8 b3
      const uint32_t s0 = b2 ? z[2 * q][0] : z[2 * q + 1][0];
      const uint32_t s1 = b2 ? z[2 * q][1] : z[2 * q + 1][1];
      const uint32_t r0 = (uint32_t)__builtin_amdgcn_ds_swizzle((int)s0, 0x101F);
      const uint32_t r3 = (uint32_t)__builtin_amdgcn_ds_swizzle((int)s1, 0x101F);
      const uint4 w = b2 ? uint4{r0, r3, z[2 * q + 1][0], z[2 * q + 1][1]}
                         : uint4{z[2 * q][0], z[2 * q][1], r0, r3};
      const int64_t c = 16 * (2 * q + (int)b2) + 8 * (int)b3;
      if (row >= g.M) continue;
      const bool whole = c + 8 <= g.N && (g.split <= 0 || c + 8 <= g.split || c >= g.split);
      if (vec && whole) {
        T* dst = g.split > 0 && c >= g.split
                     ? static_cast<T*>(g.out2) + row * g.ldo2 + (c - g.split)
                     : static_cast<T*>(g.out) + row * g.ldo + c;
        *reinterpret_cast<uint4*>(dst) = w;
      } else {
        T e[8];
        __builtin_memcpy(e, &w, 16);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (c + j < g.N) {
            if (g.split > 0 && c + j >= g.split)
              static_cast<T*>(g.out2)[row * g.ldo2 + (c + j - g.split)] = e[j];
            else
              static_cast<T*>(g.out)[row * g.ldo + c + j] = e[j];
          }
      }
    }
  }
}

// Through LDS: the wave writes its 16 MT rows x 16 NT columns (already in
// the output type) to its own region, then each lane reads back whole
// 16-byte pieces of rows, so one store instruction covers 1 KB of whole
// row pieces instead of 64-byte pieces of four rows.  A piece is stored
// whole when it lies inside the output, on one side of the split column,
// and both outputs allow 16-byte accesses; otherwise element by element.
// For 128-column tiles, piece p of local row lr sits at piece
// p ^ (((lr >> 2) & 3) << SH) of the row in LDS: the four rows one write
// instruction touches then fall on different banks (narrower tiles keep
// the plain order).  Only this wave's region is touched, so no workgroup
// barrier is needed once every wave is past the last read of the ring.
template <typename T, int MT, int NT>
__device__ __forceinline__ void store_staged(const GemmArgs& g, int64_t row0, int64_t n0,
                                             const f32x4 (&acc)[MT][NT], T* region) {
  constexpr int BN = 16 * NT, EPL = Mma<T>::EPL, PR = BN / EPL, ROWS = 16 * MT;
  constexpr int SH = NT == 8 ? (EPL == 4 ? 2 : 1) : 0;  // log2 pieces per 16 columns
  constexpr int SW = NT == 8 ? 3 : 0;                    // row bits that pick the swizzle
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int lr = mt * 16 + 4 * (lane >> 4) + r;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int col = nt * 16 + (lane & 15);
        const int pp = (col / EPL) ^ (((lr >> 2) & SW) << SH);
        region[lr * BN + pp * EPL + col % EPL] = Mma<T>::from_f(acc[mt][nt][r]);
      }
    }
  // the region is written as T and read back as 16-byte vectors: keep the
  // compiler from moving a read above a write (the wave's LDS accesses then
  // complete in program order)
  asm volatile("" ::: "memory");
  const size_t es = sizeof(T);
  const bool vec = (reinterpret_cast<uintptr_t>(g.out) & 15) == 0 && (g.ldo * es) % 16 == 0 &&
                   (g.split <= 0 || ((reinterpret_cast<uintptr_t>(g.out2) & 15) == 0 &&
                                     (g.ldo2 * es) % 16 == 0));
  const uint4* src = reinterpret_cast<const uint4*>(region);
#pragma unroll
  for (int i = 0; i < (ROWS * PR + 63) / 64; ++i) {
    const int k = i * 64 + lane, lr = k / PR, p = k % PR;
    if (k >= ROWS * PR) break;
    const uint4 v = src[lr * PR + (p ^ (((lr >> 2) & SW) << SH))];
    const int64_t row = row0 + lr, c = n0 + (int64_t)p * EPL;
    if (row >= g.M) continue;
    const bool whole = c + EPL <= g.N && (g.split <= 0 || c + EPL <= g.split || c >= g.split);
    if (vec && whole) {
      T* dst = g.split > 0 && c >= g.split
                   ? static_cast<T*>(g.out2) + row * g.ldo2 + (c - g.split)
                   : static_cast<T*>(g.out) + row * g.ldo + c;
      *reinterpret_cast<uint4*>(dst) = v;
    } else {
      T e[EPL];
      __builtin_memcpy(e, &v, 16);
#pragma unroll
      for (int j = 0; j < EPL; ++j)
        if (c + j < g.N) {
          if (g.split > 0 && c + j >= g.split)
            static_cast<T*>(g.out2)[row * g.ldo2 + (c + j - g.split)] = e[j];
          else
            static_cast<T*>(g.out)[row * g.ldo + c + j] = e[j];
        }
    }
  }
}

// staged stores need room in the ring for every wave's rows (kStaged), or
// at least for 16 rows of every wave, staged one 16-row slab at a time
template <typename T, int MT, int NT, typename R>
constexpr bool kStaged =
    (size_t)(R::THREADS / 64) * 16 * MT * 16 * NT * sizeof(T) <= R::LDS_BYTES;
template <typename T, int NT, typename R>
constexpr bool kStagedSlab = (size_t)(R::THREADS / 64) * 16 * 16 * NT * sizeof(T) <= R::LDS_BYTES;

template <typename T, int MT, int NT, typename R>
__device__ __forceinline__ void store_tile(const GemmArgs& g, int64_t row0, int64_t n0,
                                           const f32x4 (&acc)[MT][NT], uint4* ring) {
  const int wave = threadIdx.x >> 6;
  if constexpr (kStaged<T, MT, NT, R>) {
    store_staged<T, MT, NT>(g, row0, n0, acc,
                            reinterpret_cast<T*>(ring) + (size_t)wave * 16 * MT * 16 * NT);
  } else if constexpr (kStagedSlab<T, NT, R>) {
    T* region = reinterpret_cast<T*>(ring) + (size_t)wave * 16 * 16 * NT;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      // the previous slab's read-back stays ahead of this slab's writes
      asm volatile("" ::: "memory");
      store_staged<T, 1, NT>(g, row0 + mt * 16, n0,
                             reinterpret_cast<const f32x4(&)[1][NT]>(acc[mt]), region);
    }
  } else {
    store_direct<T, MT, NT>(g, row0, n0, acc);
  }
}

// PLAIN / CONCAT
template <typename T, int MT, int NT, typename R>
__global__ __launch_bounds__(R::THREADS) void k_gemm(GemmArgs g) {
  __shared__ uint4 ring[R::RING_SLOTS];
  const int wave = threadIdx.x >> 6;
  const int64_t tile0 = (int64_t)blockIdx.x * R::BM;
  const int64_t n0 = (int64_t)blockIdx.y * R::BN;
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  R::phase(static_cast<const T*>(g.a), g.lda, g.M, g.K, static_cast<const T*>(g.wt), g.kp, tile0,
           n0, ring, acc);
  if (g.mode == SAGA_GEMM_CONCAT)
    R::phase(static_cast<const T*>(g.a2), g.lda2, g.M, g.K2, static_cast<const T*>(g.wt2), g.kp2,
             tile0, n0, ring, acc);
  const int64_t row0 = tile0 + wave * MT * 16;
  finish_tile(g, row0, n0, acc);
  store_tile<T, MT, NT, R>(g, row0, n0, acc, ring);
}

// bfloat16 PLAIN with the weights resident: one workgroup per CU holds
// all of W^T for its 128 output columns in LDS (k in half chunks of 32,
// column n = 16 t + r: piece p of 8 k at slot ((h * 8 + t) * 4 + p) * 16 + r,
// so the 16 lanes that read one piece of 16 columns read 256 contiguous
// bytes, free of bank conflicts), loaded once.  Each wave
// then streams its own 16 MT-row tiles (tile q = wave id, wave id + all
// waves, ...) through D register slots of A chunks; the stream runs on
// across tiles, so the next tile's first chunks are in flight during the
// last chunks and the epilogue of the current one.  No workgroup barrier
// after the weights land, and only A loads on the vmcnt counter, so a wait
// for one chunk never drains the chunks behind it.  The LDS being taken,
// the epilogue stores through lane exchanges (store_shuffled).
constexpr int kResHalfChunks = 19;  // half chunks of 32 k: K <= 608, 152 KB of LDS

template <int MT, int NW, int D>
__global__ __launch_bounds__(64 * NW) void k_gemm_bres(GemmArgs g) {
  typedef uint16_t T;
  typedef RegA<T, MT, 8, 2, NW> R;
  typedef typename Mma<T>::Frag Frag;
  constexpr int NT = 8, KC = Mma<T>::KC;
  static_assert(D >= 2 && D <= 8, "A slots");
  __shared__ uint4 wres[kResHalfChunks * 128 * 4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const T* A = static_cast<const T*>(g.a);
  const T* Wt = static_cast<const T*>(g.wt);
  const int hc = (int)((g.K + 31) / 32);  // half chunks held (<= kResHalfChunks, checked by the host)
  // weights: slot s of half chunk h, column n, piece p
  {
    const int slots = hc * 128 * 4;
    for (int s0 = wave * 64; s0 < slots; s0 += NW * 64) {
      const int s = s0 + lane, h = s / 512, p = (s / 16) % 4;
      // columns past N (not packed when N < 128) repeat column N - 1; their
      // outputs are never stored
      const int n = min((s / 64) % 8 * 16 + s % 16, (int)g.N - 1);
      __builtin_amdgcn_global_load_lds(Wt + (int64_t)n * g.kp + h * 32 + p * 8, (lds_ptr)(wres + s0),
                                       16, 0, 0);
    }
    wait_vm<0>();
    ring_barrier();
  }
  const int nch = (int)((g.K + KC - 1) / KC);
  const int64_t ntile = (g.M + 16 * MT - 1) / (16 * MT);
  const int64_t gw = (int64_t)blockIdx.x * NW + wave, stride = (int64_t)gridDim.x * NW;
  if (gw >= ntile) return;
  const int64_t mytiles = (ntile - gw + stride - 1) / stride;
  const int64_t total = mytiles * nch;  // chunks in this wave's stream
  // the stream's read position (tile q_pf, chunk c_pf) and compute position
  // (tile q_cur, chunk c_cur), advanced one chunk at a time
  int64_t q_pf = gw, q_cur = gw;
  int c_pf = 0, c_cur = 0;
  int64_t off_pf[MT];
  R::row_offsets(nullptr, g.lda, g.M, q_pf * 16 * MT, off_pf);
  auto issue_next = [&](Frag (&a)[2][MT]) {
    R::load_a(A, off_pf, g.K, (int64_t)c_pf * KC, a);
    if (++c_pf == nch) {  // rows of tiles past the last are clamped to row M - 1
      c_pf = 0;
      q_pf += stride;
      R::row_offsets(nullptr, g.lda, g.M, q_pf * 16 * MT, off_pf);
    }
  };
  Frag a[D][2][MT];
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // chunk i of the stream from register slot U; FULL: the read of chunk
  // i + D - 1 exists (the steady state: no conditional loads, so the
  // compiler's waits count exactly the D - 1 chunks in flight)
  auto step = [&](auto u_c, auto full_c, int64_t i) {
    constexpr int U = decltype(u_c)::value;
    constexpr bool FULL = decltype(full_c)::value;
    if constexpr (FULL) {
      issue_next(a[(U + D - 1) % D]);
    } else {
      if (i >= total) return;
      if (i + D - 1 < total) issue_next(a[(U + D - 1) % D]);
    }
    const int c = c_cur;
    if (c == nch - 1) R::mask(g.K, (int64_t)c * KC, a[U]);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int hh = 2 * c + h;
      if (hh >= hc) break;  // past K: the A values there are zero, the weights not held
      Frag b[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const uint4 v = wres[((hh * 8 + nt) * 4 + lg) * 16 + lr];
        __builtin_memcpy(&b[nt], &v, 16);
      }
      __builtin_amdgcn_sched_barrier(0);  // every fragment read ahead of the MFMAs
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[U][h][mt], b[nt], acc[mt][nt], 0, 0, 0);
    }
    if (++c_cur == nch) {
      const int64_t row0 = q_cur * 16 * MT;
      finish_tile(g, row0, 0, acc);
      store_shuffled<MT>(g, row0, acc);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      c_cur = 0;
      q_cur += stride;
    }
  };
  using T1 = std::true_type;
  using T0 = std::false_type;
  int64_t i0 = 0;
  if (total >= 2 * D - 1) {
    // the first D - 1 chunks, unconditionally: the steady loop below is
    // entered only from here, with exactly D - 1 chunks in flight
#pragma unroll
    for (int j = 0; j < D - 1; ++j) issue_next(a[j]);
    // steady state: every step's read exists (i + D - 1 < total)
    for (; i0 + 2 * D - 1 <= total; i0 += D) {
      step(std::integral_constant<int, 0>{}, T1{}, i0);
      step(std::integral_constant<int, 1>{}, T1{}, i0 + 1);
      if constexpr (D > 2) step(std::integral_constant<int, 2>{}, T1{}, i0 + 2);
      if constexpr (D > 3) step(std::integral_constant<int, 3>{}, T1{}, i0 + 3);
      if constexpr (D > 4) step(std::integral_constant<int, 4>{}, T1{}, i0 + 4);
      if constexpr (D > 5) step(std::integral_constant<int, 5>{}, T1{}, i0 + 5);
      if constexpr (D > 6) step(std::integral_constant<int, 6>{}, T1{}, i0 + 6);
      if constexpr (D > 7) step(std::integral_constant<int, 7>{}, T1{}, i0 + 7);
    }
  } else {
#pragma unroll
    for (int j = 0; j < D - 1; ++j)
      if (j < total) issue_next(a[j]);
  }
  // the last chunks, fewer or no reads
  for (; i0 < total; i0 += D) {
    step(std::integral_constant<int, 0>{}, T0{}, i0);
    step(std::integral_constant<int, 1>{}, T0{}, i0 + 1);
    if constexpr (D > 2) step(std::integral_constant<int, 2>{}, T0{}, i0 + 2);
    if constexpr (D > 3) step(std::integral_constant<int, 3>{}, T0{}, i0 + 3);
    if constexpr (D > 4) step(std::integral_constant<int, 4>{}, T0{}, i0 + 4);
    if constexpr (D > 5) step(std::integral_constant<int, 5>{}, T0{}, i0 + 5);
    if constexpr (D > 6) step(std::integral_constant<int, 6>{}, T0{}, i0 + 6);
    if constexpr (D > 7) step(std::integral_constant<int, 7>{}, T0{}, i0 + 7);
  }
}

// GRU: acc1 = a w (input gates), acc2 = a2 w2 (hidden gates), column blocks
// (r, z, n) of width F = NT3 * 16; hidden state h = a2
template <typename T, int NT3, int S>
__global__ __launch_bounds__(kThreads) void k_gemm_gru(GemmArgs g) {
  constexpr int NT = 3 * NT3;
  typedef RegA<T, 1, NT, S> R;
  __shared__ uint4 ring[R::RING_SLOTS];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t tile0 = (int64_t)blockIdx.x * R::BM;
  f32x4 acc1[1][NT], acc2[1][NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    acc1[0][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc2[0][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const T* h = static_cast<const T*>(g.a2);
  R::phase(static_cast<const T*>(g.a), g.lda, g.M, g.K, static_cast<const T*>(g.wt), g.kp, tile0,
           0, ring, acc1);
  R::phase(h, g.lda2, g.M, g.K2, static_cast<const T*>(g.wt2), g.kp2, tile0, 0, ring, acc2);
  const int F = NT3 * 16;
  const int64_t row0 = tile0 + wave * 16;
  T* out = static_cast<T*>(g.out);
  // biases and previous states are all loaded before the first store (a
  // load after a store the compiler cannot tell apart from it would wait)
  float bi[3][NT3], bh[3][NT3], hp[4][NT3];
#pragma unroll
  for (int t = 0; t < NT3; ++t) {
    const int c = t * 16 + (lane & 15);
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      bi[q][t] = g.bias ? g.bias[q * F + c] : 0.f;
      bh[q][t] = g.bias2 ? g.bias2[q * F + c] : 0.f;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = row0 + 4 * (lane >> 4) + r;
      hp[r][t] = row < g.M ? Mma<T>::to_f(h[row * g.lda2 + c]) : 0.f;
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t row = row0 + 4 * (lane >> 4) + r;
    if (row >= g.M) continue;
#pragma unroll
    for (int t = 0; t < NT3; ++t) {
      const int c = t * 16 + (lane & 15);
      const float rr = sigmoidf_(acc1[0][t][r] + bi[0][t] + acc2[0][t][r] + bh[0][t]);
      const float zz = sigmoidf_(acc1[0][t + NT3][r] + bi[1][t] + acc2[0][t + NT3][r] + bh[1][t]);
      const float nn =
          tanhf(acc1[0][t + 2 * NT3][r] + bi[2][t] + rr * (acc2[0][t + 2 * NT3][r] + bh[2][t]));
      out[row * g.ldo + c] = Mma<T>::from_f((1.0f - zz) * nn + zz * hp[r][t]);
    }
  }
}

// Grouped: row q of the output is row arow[q] of A times the weight of the
// group whose row range holds q (R-GCN's per-relation transform of the
// distinct (relation, source) pairs).  Group ranges are whole tiles, so a
// tile finds its group by a binary search of grp_ptr and multiplies by that
// group's packed weight; tiles from grp_ptr[groups] on are idle.  Rows whose
// map entry is negative (range padding) are written as zeros.
template <typename T, int MT, int NT, typename R>
__global__ __launch_bounds__(R::THREADS) void k_gemm_grouped(GemmArgs g) {
  static_assert(R::BM == kRelTile, "grouped tiles must match the row-range padding");
  __shared__ uint4 ring[R::RING_SLOTS];
  if ((g.err1 && *g.err1) || (g.err2 && *g.err2)) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t tile0 = (int64_t)blockIdx.x * R::BM;
  const int64_t rows = g.grp_ptr[g.groups];
  if (tile0 >= rows) return;
  int lo = 0, hi = g.groups;  // grp_ptr[lo] <= tile0 < grp_ptr[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (g.grp_ptr[mid] <= tile0) lo = mid;
    else hi = mid;
  }
  const int64_t n0 = (int64_t)blockIdx.y * R::BN;
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  R::phase(static_cast<const T*>(g.a), g.lda, g.M, g.K,
           static_cast<const T*>(g.wt) + (int64_t)lo * g.wt_group_stride, g.kp, tile0, n0, ring,
           acc, g.arow);
  const int64_t row0 = tile0 + wave * MT * 16;
  // rows of range padding (map entry < 0) are written as zeros
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (g.arow[row0 + mt * 16 + 4 * (lane >> 4) + r] < 0) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt][r] = 0.0f;
      }
  store_tile<T, MT, NT, R>(g, row0, n0, acc, ring);
}

// Wt[grp][n][k] = W[grp K + k][n] for n < N, k < K, else 0; each group's
// packed weight is Np x Kp with ld Kp
template <typename T>
__global__ __launch_bounds__(kThreads) void k_pack_wt_grouped(const T* __restrict__ W,
                                                              int64_t ldw, int64_t K, int64_t N,
                                                              int groups, T* __restrict__ Wt,
                                                              int64_t Kp, int64_t Np) {
  const int64_t per = Np * Kp, total = per * groups;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t grp = i / per, j = i - grp * per;
    const int64_t n = j / Kp, k = j - n * Kp;
    Wt[i] = (n < N && k < K) ? W[(grp * K + k) * ldw + n] : T(0);
  }
}

// ---------------------------------------------------------------------------
// host side: tiling choice, weight packing, launch
// ---------------------------------------------------------------------------
struct Tiling {
  int mt, nt, stages;
  bool ring_a;  // A through the LDS ring (Ring) instead of registers (RegA)
  int nw = 4;   // waves per workgroup (RegA)
};

#ifdef SAGA_SWEEP_BUILD
// A sweep build reads SAGA_GEMM_CFG to override the tile shape of the N <= 128 kernels for tuning:
// "aMxS" = A through registers, M = rows per wave / 16, S stages;
// "rMxS" = A through the LDS ring
Tiling cfg_override(Tiling t) {
  static const char* e = getenv("SAGA_GEMM_CFG");
  if (!e) return t;
  static const struct { const char* name; Tiling t; } table[] = {
      {"r2x2", {2, 8, 2, true}}, {"r2x4", {2, 8, 4, true}}, {"a2x4", {2, 8, 4, false}},
      {"a2x3", {2, 8, 3, false}}, {"a4x3", {4, 8, 3, false}}, {"a4x2", {4, 8, 2, false}},
      {"a1x4", {1, 8, 4, false}}, {"a2x3w8", {2, 8, 3, false, 8}}, {"a2x2w8", {2, 8, 2, false, 8}},
      {"a2x4w8", {2, 8, 4, false, 8}}, {"a1x4w8", {1, 8, 4, false, 8}},
      {"a1x4w16", {1, 8, 4, false, 16}}, {"a1x3w16", {1, 8, 3, false, 16}},
      {"a1x3w8", {1, 8, 3, false, 8}}};
  for (const auto& x : table)
    if (!strcmp(e, x.name)) return x.t;
  return t;
}
#else
Tiling cfg_override(Tiling t) { return t; }
#endif

// k chunks of a K-long operand
int64_t chunks(int dtype, int64_t K) {
  const int64_t kc = dtype == SAGA_BF16 ? Mma<uint16_t>::KC : Mma<float>::KC;
  return (K + kc - 1) / kc;
}

Tiling choose(int dtype, int mode, int64_t N, int64_t K) {
  if (mode == SAGA_GEMM_GRU) return Tiling{1, (int)(N / 16), 4, false};
  const int64_t nt = (N + 15) / 16;
  // narrow tiles: with at most four k chunks two stages suffice (the
  // registers two more A slots would hold buy occupancy instead; measured
  // on the 2^21 x 128 x 41 transform: 0.437 -> 0.414 ms fp32, 0.175 ->
  // 0.162 ms bf16)
  if (nt <= 5) return Tiling{2, (int)nt, chunks(dtype, K) <= 4 ? 2 : 4, false};
  // 128-column tiles (more columns: several tiles along N), measured best
  // on the 2^21 x 602 x 128 transform and on 131072 x 512 x 256
  return cfg_override(dtype == SAGA_BF16 ? Tiling{1, 8, 4, false, 8} : Tiling{2, 8, 2, true});
}

int kc_of(int dtype) { return dtype == SAGA_BF16 ? Mma<uint16_t>::KC : Mma<float>::KC; }

struct Packed {
  int64_t np, kp, kp2;
  size_t off2, bytes;
};

Packed packed_layout(int dtype, int mode, int64_t N, int64_t K, int64_t K2) {
  const Tiling t = choose(dtype, mode, N, K);
  const int64_t bn = 16 * t.nt, kc = kc_of(dtype);
  const size_t es = dtype == SAGA_BF16 ? 2 : 4;
  Packed p;
  p.np = (N + bn - 1) / bn * bn;
  p.kp = (K + kc - 1) / kc * kc;
  p.kp2 = mode == SAGA_GEMM_PLAIN ? 0 : (K2 + kc - 1) / kc * kc;
  const size_t b1 = ((size_t)p.np * p.kp * es + 255) / 256 * 256;
  p.off2 = b1;
  p.bytes = b1 + ((size_t)p.np * p.kp2 * es + 255) / 256 * 256;
  return p;
}

template <typename T, int MT, int NT, typename R>
hipError_t launch_plain(const GemmArgs& g, hipStream_t st) {
  static_assert(R::LDS_BYTES <= 160 * 1024, "LDS ring too large");
  dim3 grid((unsigned)((g.M + R::BM - 1) / R::BM), (unsigned)((g.N + R::BN - 1) / R::BN));
  hipLaunchKernelGGL((k_gemm<T, MT, NT, R>), grid, dim3(R::THREADS), 0, st, g);
  return hipGetLastError();
}

template <typename T, int NT>
hipError_t launch_nt(const GemmArgs& g, const Tiling& t, hipStream_t st) {
  if constexpr (NT == 8) {
    if (t.ring_a) {
      if (t.stages == 2) return launch_plain<T, 2, 8, Ring<T, 2, 8, 2>>(g, st);
      return launch_plain<T, 2, 8, Ring<T, 2, 8, 4>>(g, st);
    }
    if (t.nw == 16) {
      if (t.stages == 3) return launch_plain<T, 1, 8, RegA<T, 1, 8, 3, 16>>(g, st);
      return launch_plain<T, 1, 8, RegA<T, 1, 8, 4, 16>>(g, st);
    }
    if (t.nw == 8) {
      if (t.mt == 1 && t.stages == 3) return launch_plain<T, 1, 8, RegA<T, 1, 8, 3, 8>>(g, st);
      if (t.mt == 1) return launch_plain<T, 1, 8, RegA<T, 1, 8, 4, 8>>(g, st);
      if (t.stages == 2) return launch_plain<T, 2, 8, RegA<T, 2, 8, 2, 8>>(g, st);
      if (t.stages == 4) return launch_plain<T, 2, 8, RegA<T, 2, 8, 4, 8>>(g, st);
      return launch_plain<T, 2, 8, RegA<T, 2, 8, 3, 8>>(g, st);
    }
    if (t.mt == 1) return launch_plain<T, 1, 8, RegA<T, 1, 8, 4>>(g, st);
    if (t.mt == 4 && t.stages == 2) return launch_plain<T, 4, 8, RegA<T, 4, 8, 2>>(g, st);
    if (t.mt == 4) return launch_plain<T, 4, 8, RegA<T, 4, 8, 3>>(g, st);
    if (t.stages == 3) return launch_plain<T, 2, 8, RegA<T, 2, 8, 3>>(g, st);
  }
  if (t.stages == 2) return launch_plain<T, 2, NT, RegA<T, 2, NT, 2>>(g, st);
  return launch_plain<T, 2, NT, RegA<T, 2, NT, 4>>(g, st);
}

// weight-resident bfloat16 kernel: one workgroup per CU (its LDS holds the
// weights), or fewer when there are fewer tiles than waves
template <int MT, int NW, int D>
hipError_t launch_bres(const GemmArgs& g, hipStream_t st) {
  static int cus = [] {
    int dev = 0, n = 256;
    if (hipGetDevice(&dev) == hipSuccess)
      (void)hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    return n > 0 ? n : 256;
  }();
  const int64_t tiles = (g.M + 16 * MT - 1) / (16 * MT);
  const int64_t wgs = std::max<int64_t>(1, std::min<int64_t>(cus, (tiles + NW - 1) / NW));
  hipLaunchKernelGGL((k_gemm_bres<MT, NW, D>), dim3((unsigned)wgs), dim3(64 * NW), 0, st, g);
  return hipGetLastError();
}

// The weight-resident kernel takes bfloat16 PLAIN products with 80 < N <=
// 128 (narrower outputs use the narrow tiles) and 192 <= K <= 608.  On
// 2^21 rows x 128 columns against the streamed tiles: 0.32 / 0.35 ms at
// K = 192 (one 16-row tile per wave), 0.37 / 0.42 ms at K = 256, 0.49 /
// 0.55 at 384 and 0.69 / 0.80 at 602 (two tiles per wave, three A slots:
// as fast as four, which spill registers); at K = 128 the streamed tiles
// are as fast.  A sweep build reads SAGA_GEMM_BRES to override the shape
// ("MxWxD": M x 16 rows per wave, W waves, D A chunks in registers; "off":
// the streamed tiles).
hipError_t maybe_bres(const GemmArgs& g, hipStream_t st, bool* used) {
  *used = false;
  if (g.dtype != SAGA_BF16 || g.mode != SAGA_GEMM_PLAIN || g.N > 128 || g.K > 32 * kResHalfChunks)
    return hipSuccess;
#ifdef SAGA_SWEEP_BUILD
  static const char* e = getenv("SAGA_GEMM_BRES");
  const char* cfg = e ? e : g.N <= 80 || g.K < 192 ? "off" : g.K < 256 ? "1x8x4" : "2x8x3";
  *used = true;
  if (!strcmp(cfg, "1x8x4")) return launch_bres<1, 8, 4>(g, st);
  if (!strcmp(cfg, "2x8x4")) return launch_bres<2, 8, 4>(g, st);
  if (!strcmp(cfg, "2x8x3")) return launch_bres<2, 8, 3>(g, st);
  if (!strcmp(cfg, "1x16x3")) return launch_bres<1, 16, 3>(g, st);
  if (!strcmp(cfg, "1x8x6")) return launch_bres<1, 8, 6>(g, st);
  *used = false;
  return hipSuccess;
#else
  if (g.N <= 80 || g.K < 192) return hipSuccess;
  *used = true;
  return g.K < 256 ? launch_bres<1, 8, 4>(g, st) : launch_bres<2, 8, 3>(g, st);
#endif
}

template <typename T>
hipError_t dispatch(const GemmArgs& g, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    bool used = false;
    const hipError_t e = maybe_bres(g, st, &used);
    if (used || e != hipSuccess) return e;
  }
  const Tiling t = choose(g.dtype, g.mode, g.N, g.mode == SAGA_GEMM_CONCAT ? g.K + g.K2 : g.K);
  if (g.mode == SAGA_GEMM_GRU) {
    dim3 grid((unsigned)((g.M + 63) / 64));
    // two stages when both products have at most four k chunks (as for the
    // narrow plain tiles)
    const bool two = chunks(g.dtype, std::max(g.K, g.K2)) <= 4;
#define SAGA_GRU(N3)                                                                     \
  if (two) hipLaunchKernelGGL((k_gemm_gru<T, N3, 2>), grid, dim3(kThreads), 0, st, g);  \
  else hipLaunchKernelGGL((k_gemm_gru<T, N3, 4>), grid, dim3(kThreads), 0, st, g)
    switch (t.nt) {
      case 3: SAGA_GRU(1); break;
      case 6: SAGA_GRU(2); break;
      case 9: SAGA_GRU(3); break;
      case 12: SAGA_GRU(4); break;
      default: return hipErrorInvalidValue;
    }
#undef SAGA_GRU
    return hipGetLastError();
  }
  switch (t.nt) {
    case 1: return launch_nt<T, 1>(g, t, st);
    case 2: return launch_nt<T, 2>(g, t, st);
    case 3: return launch_nt<T, 3>(g, t, st);
    case 4: return launch_nt<T, 4>(g, t, st);
    case 5: return launch_nt<T, 5>(g, t, st);
    default: return launch_nt<T, 8>(g, t, st);
  }
}

template <typename T>
hipError_t pack(const void* w, int64_t ldw, int64_t K, int64_t N, void* wt, int64_t kp,
                int64_t np, hipStream_t st) {
  const int64_t total = np * kp;
  const unsigned blocks = (unsigned)std::min<int64_t>((total + kThreads - 1) / kThreads, 2048);
  hipLaunchKernelGGL((k_pack_wt<T>), dim3(blocks), dim3(kThreads), 0, st, static_cast<const T*>(w),
                     ldw, K, N, static_cast<T*>(wt), kp, np);
  return hipGetLastError();
}

// grouped GEMM tiling: 128-row tiles (RegA, 2 x 16 rows per wave, 4 waves,
// 4 stages), up to 128 columns per tile
inline int grouped_nt(int64_t N) { return (int)std::min<int64_t>(8, (N + 15) / 16); }

template <typename T, int NT>
hipError_t launch_grouped_nt(const GemmArgs& g, hipStream_t st) {
  auto go = [&](auto r) {
    typedef decltype(r) R;
    dim3 grid((unsigned)(g.M / R::BM), (unsigned)((g.N + R::BN - 1) / R::BN));
    hipLaunchKernelGGL((k_gemm_grouped<T, 2, NT, R>), grid, dim3(R::THREADS), 0, st, g);
    return hipGetLastError();
  };
  // two stages for at most four k chunks, as for the plain narrow tiles
  if (chunks(g.dtype, g.K) <= 4) return go(RegA<T, 2, NT, 2>{});
  return go(RegA<T, 2, NT, 4>{});
}

template <typename T>
hipError_t dispatch_grouped(const GemmArgs& g, hipStream_t st) {
  switch (grouped_nt(g.N)) {
    case 1: return launch_grouped_nt<T, 1>(g, st);
    case 2: return launch_grouped_nt<T, 2>(g, st);
    case 3: return launch_grouped_nt<T, 3>(g, st);
    case 4: return launch_grouped_nt<T, 4>(g, st);
    case 5: return launch_grouped_nt<T, 5>(g, st);
    case 6: return launch_grouped_nt<T, 6>(g, st);
    case 7: return launch_grouped_nt<T, 7>(g, st);
    default: return launch_grouped_nt<T, 8>(g, st);
  }
}

void grouped_packed(int dtype, int64_t N, int64_t K, int64_t* np, int64_t* kp) {
  const int64_t bn = 16 * grouped_nt(N), kc = kc_of(dtype);
  *np = (N + bn - 1) / bn * bn;
  *kp = (K + kc - 1) / kc * kc;
}

}  // namespace

size_t gemm_workspace_bytes(int dtype, int mode, int64_t N, int64_t K, int64_t K2) {
  return packed_layout(dtype, mode, N, K, K2).bytes;
}

hipError_t launch_gemm(const GemmArgs& g0, hipStream_t st) {
  if (g0.M == 0) return hipSuccess;
  const Packed pk = packed_layout(g0.dtype, g0.mode, g0.N, g0.K, g0.K2);
  if (!g0.ws || g0.ws_bytes < pk.bytes) return hipErrorInvalidValue;
  GemmArgs g = g0;
  char* ws = static_cast<char*>(g.ws);
  g.wt = ws;
  g.kp = pk.kp;
  g.wt2 = pk.kp2 ? ws + pk.off2 : nullptr;
  g.kp2 = pk.kp2;
  const bool bf = g.dtype == SAGA_BF16;
  hipError_t e = bf ? pack<uint16_t>(g.w, g.ldw, g.K, g.N, ws, pk.kp, pk.np, st)
                    : pack<float>(g.w, g.ldw, g.K, g.N, ws, pk.kp, pk.np, st);
  if (e == hipSuccess && pk.kp2)
    e = bf ? pack<uint16_t>(g.w2, g.ldw2, g.K2, g.N, ws + pk.off2, pk.kp2, pk.np, st)
           : pack<float>(g.w2, g.ldw2, g.K2, g.N, ws + pk.off2, pk.kp2, pk.np, st);
  if (e != hipSuccess) return e;
  return bf ? dispatch<uint16_t>(g, st) : dispatch<float>(g, st);
}

size_t gemm_grouped_workspace_bytes(int dtype, int groups, int64_t N, int64_t K) {
  int64_t np, kp;
  grouped_packed(dtype, N, K, &np, &kp);
  const size_t es = dtype == SAGA_BF16 ? 2 : 4;
  return ((size_t)groups * np * kp * es + 255) / 256 * 256;
}

hipError_t launch_gemm_grouped(const GemmArgs& g0, hipStream_t st) {
  if (g0.M == 0) return hipSuccess;
  if (g0.M % kRelTile != 0 || g0.groups < 1 || !g0.arow || !g0.grp_ptr) return hipErrorInvalidValue;
  if (!g0.ws || g0.ws_bytes < gemm_grouped_workspace_bytes(g0.dtype, g0.groups, g0.N, g0.K))
    return hipErrorInvalidValue;
  GemmArgs g = g0;
  int64_t np, kp;
  grouped_packed(g.dtype, g.N, g.K, &np, &kp);
  g.wt = g.ws;
  g.kp = kp;
  g.wt_group_stride = np * kp;
  const bool bf = g.dtype == SAGA_BF16;
  const int64_t total = np * kp * g.groups;
  const unsigned blocks = (unsigned)std::min<int64_t>((total + kThreads - 1) / kThreads, 4096);
  if (bf)
    hipLaunchKernelGGL((k_pack_wt_grouped<uint16_t>), dim3(blocks), dim3(kThreads), 0, st,
                       static_cast<const uint16_t*>(g.w), g.ldw, g.K, g.N, g.groups,
                       static_cast<uint16_t*>(g.ws), kp, np);
  else
    hipLaunchKernelGGL((k_pack_wt_grouped<float>), dim3(blocks), dim3(kThreads), 0, st,
                       static_cast<const float*>(g.w), g.ldw, g.K, g.N, g.groups,
                       static_cast<float*>(g.ws), kp, np);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return bf ? dispatch_grouped<uint16_t>(g, st) : dispatch_grouped<float>(g, st);
}

}  // namespace saga
