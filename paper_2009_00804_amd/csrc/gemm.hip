// ApplyVertex: the dense per-vertex transform (Sec. 3.2 "ApplyVertex" of
// the paper: all vertices batched into one GEMM, Table III) on the CDNA4
// matrix cores, with the layer's epilogue fused (degree row scaling, bias,
// activation, the two-operand concat form [a | a2][w ; w2], and the GRU
// gate math of GGNN's ApplyVertex, Fig. 2).
//
// Tiling: a workgroup of 4 waves owns BM = 4 * MT * 16 rows and NT * 16
// columns.  A wave computes MT x NT tiles of 16 x 16 with
//   float32 : v_mfma_f32_16x16x4f32   (4 k per instruction)
//   bfloat16: v_mfma_f32_16x16x32_bf16 (32 k per instruction, gfx950)
// A fragments come straight from global memory as 16-byte row slices (lane
// l reads row l % 16 at k offset (l / 16) * EPL, which is the operand layout
// up to a permutation of k that A and B share); the weight chunk of KC rows
// is staged transposed in LDS so each lane reads its B fragment as one
// 16-byte LDS load.
#include <cstdlib>

#include "saga_device.h"
#include "saga_internal.h"

namespace saga {
namespace {

constexpr int kThreads = 256;

template <typename T> struct Mma;

template <> struct Mma<float> {
  static constexpr int EPL = 4;     // elements per lane per fragment
  static constexpr int KSTEP = 16;  // k covered by one fragment set
  static constexpr int KC = 32;     // k rows of W staged per LDS chunk
  static constexpr int PAD = 4;
  typedef f32x4 Frag;
  __device__ __forceinline__ static void mma(const Frag& a, const Frag& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
  }
  __device__ __forceinline__ static Frag zero() { return Frag{0.f, 0.f, 0.f, 0.f}; }
  __device__ __forceinline__ static float to_f(float x) { return x; }
  __device__ __forceinline__ static float from_f(float x) { return x; }
};

template <> struct Mma<uint16_t> {
  static constexpr int EPL = 8;
  static constexpr int KSTEP = 32;
  static constexpr int KC = 64;
  static constexpr int PAD = 8;
  typedef bf16x8 Frag;
  __device__ __forceinline__ static void mma(const Frag& a, const Frag& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static Frag zero() {
    Frag f;
    uint4 z = make_uint4(0, 0, 0, 0);
    __builtin_memcpy(&f, &z, 16);
    return f;
  }
  __device__ __forceinline__ static float to_f(uint16_t x) { return bf16_to_f32(x); }
  __device__ __forceinline__ static uint16_t from_f(float x) { return f32_to_bf16(x); }
};

// 16-byte fragment of row r, columns [k, k + EPL), zero outside [0,M) x [0,K)
template <typename T>
__device__ __forceinline__ typename Mma<T>::Frag load_a(const T* __restrict__ A, int64_t lda,
                                                        int64_t r, int64_t k, int64_t M,
                                                        int64_t K) {
  constexpr int EPL = Mma<T>::EPL;
  typename Mma<T>::Frag f = Mma<T>::zero();
  if (r < M && k < K) {
    const T* p = A + r * lda + k;
    if (k + EPL <= K) {
      __builtin_memcpy(&f, p, 16);
    } else {
      T tmp[EPL];
#pragma unroll
      for (int i = 0; i < EPL; ++i) tmp[i] = (k + i < K) ? p[i] : T(0);
      __builtin_memcpy(&f, tmp, 16);
    }
  }
  return f;
}

// ---------------------------------------------------------------------------
// Software pipeline (per workgroup, per K chunk of KC):
//   * the A fragments of chunk i+1 are loaded into registers while the MFMAs
//     of chunk i run (A streams from HBM once, straight into registers);
//   * the W rows of chunk i+1 are loaded into registers, then written
//     transposed into the other half of a double-buffered LDS tile after
//     the MFMAs of chunk i, so there is one barrier per chunk;
//   * MFMAs are issued k-step-major, then n-tile, then m-tile, so that
//     consecutive updates of one accumulator are MT*NT instructions apart.
// ---------------------------------------------------------------------------
// A K chunk of W (KC rows x BN columns) passes through registers into the
// transposed LDS tile Bt[n][k].  Thread t owns K-row group t % KG and a
// column block t / KG, so that for every column the lanes of a half-wave
// write consecutive LDS words (no bank conflicts beyond 2-way).
//   float32 : KG = KC = 32 rows, one row per thread
//   bfloat16: KG = KC / 2 = 32 row pairs, packed as one 32-bit word
template <typename T, int NT>
struct BStage {
  static constexpr int KC = Mma<T>::KC;
  static constexpr int BN = NT * 16;
  static constexpr int RPT = sizeof(T) == 4 ? 1 : 2;  // K rows per thread
  static constexpr int KG = KC / RPT;                 // 32
  static constexpr int NBLK = kThreads / KG;          // 8 column blocks
  static constexpr int CPT = (BN + NBLK - 1) / NBLK;  // columns per thread
  T v[RPT][CPT];

  __device__ __forceinline__ void load(const T* __restrict__ W, int64_t ldw, int64_t K, int64_t N,
                                       int64_t k0, int64_t n0, bool vec_ok) {
    const int kg = threadIdx.x % KG, nb = threadIdx.x / KG;
    const int64_t nbase = n0 + (int64_t)nb * CPT;
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int64_t k = k0 + (int64_t)kg * RPT + r;
      const bool kin = k < K;
      if (kin && vec_ok && (CPT * sizeof(T)) % 16 == 0 && nbase + CPT <= N && nb * CPT < BN) {
#pragma unroll
        for (int c = 0; c < CPT; c += 16 / (int)sizeof(T))
          __builtin_memcpy(&v[r][c], W + k * ldw + nbase + c, 16);
      } else {
#pragma unroll
        for (int c = 0; c < CPT; ++c)
          v[r][c] = (kin && nbase + c < N && nb * CPT + c < BN) ? W[k * ldw + nbase + c] : T(0);
      }
    }
  }
  __device__ __forceinline__ void store(T* Bt) const {
    constexpr int LDB = KC + Mma<T>::PAD;
    const int kg = threadIdx.x % KG, nb = threadIdx.x / KG;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int n = nb * CPT + c;
      if (n < BN) {
        if constexpr (RPT == 1) {
          Bt[n * LDB + kg] = v[0][c];
        } else {
          const uint32_t w = (uint32_t)v[0][c] | ((uint32_t)v[1][c] << 16);
          *reinterpret_cast<uint32_t*>(Bt + n * LDB + kg * 2) = w;
        }
      }
    }
  }
};

template <typename T, int MT>
__device__ __forceinline__ void load_a_chunk(const T* __restrict__ A, int64_t lda, int64_t M,
                                             int64_t K, int64_t row0, int64_t k0,
                                             typename Mma<T>::Frag (&af)[Mma<T>::KC / Mma<T>::KSTEP][MT]) {
  constexpr int EPL = Mma<T>::EPL;
  constexpr int NS = Mma<T>::KC / Mma<T>::KSTEP;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      af[s][mt] = load_a<T>(A, lda, row0 + mt * 16 + lr, k0 + s * Mma<T>::KSTEP + lg * EPL, M, K);
}

template <typename T, int MT, int NT>
__device__ __forceinline__ void mma_chunk(const T* Bt,
                                          const typename Mma<T>::Frag (&af)[Mma<T>::KC / Mma<T>::KSTEP][MT],
                                          f32x4 (&acc)[MT][NT]) {
  constexpr int EPL = Mma<T>::EPL;
  constexpr int KSTEP = Mma<T>::KSTEP;
  constexpr int NS = Mma<T>::KC / KSTEP;
  constexpr int LDB = Mma<T>::KC + Mma<T>::PAD;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    typename Mma<T>::Frag bf[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      __builtin_memcpy(&bf[nt], Bt + (nt * 16 + lr) * LDB + s * KSTEP + lg * EPL, 16);
    if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[s][mt][c], bf[nt][c], acc[mt][nt], 0, 0, 0);
    } else {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) Mma<T>::mma(af[s][mt], bf[nt], acc[mt][nt]);
    }
  }
}

// acc += A[row0 .. row0 + 16 MT) x W[:, n0 .. n0 + 16 NT)
//
// The A fragments of chunks ci+1 .. ci+PD-1 are in flight (registers) while
// chunk ci is multiplied; the loop is unrolled by PD so every register slot
// has a compile-time index.  The W chunk ci+1 is loaded into registers at the
// top of step ci and written (transposed) into the other LDS half after the
// MFMAs; one barrier per chunk.
template <typename T, int MT, int NT, int PD>
struct Pipe {
  typedef typename Mma<T>::Frag Frag;
  static constexpr int KC = Mma<T>::KC;
  static constexpr int NS = KC / Mma<T>::KSTEP;
  const T* A; int64_t lda; const T* W; int64_t ldw; int64_t M, N, K, row0, n0;
  bool vec_ok; int nchunks;
  T* Bt0; T* Bt1;
  BStage<T, NT> bs;

  __device__ __forceinline__ void step(int ci, Frag (&a)[NS][MT], f32x4 (&acc)[MT][NT]) {
    const bool more = ci + 1 < nchunks;
    if (more) bs.load(W, ldw, K, N, (int64_t)(ci + 1) * KC, n0, vec_ok);
    mma_chunk<T, MT, NT>((ci & 1) ? Bt1 : Bt0, a, acc);
    if (ci + PD < nchunks) load_a_chunk<T, MT>(A, lda, M, K, row0, (int64_t)(ci + PD) * KC, a);
    if (more) bs.store((ci & 1) ? Bt0 : Bt1);
    __syncthreads();
  }
};

template <typename T, int MT, int NT>
__device__ __forceinline__ void mma_phase(const T* __restrict__ A, int64_t lda,
                                          const T* __restrict__ W, int64_t ldw, int64_t M,
                                          int64_t N, int64_t K, int64_t row0, int64_t n0,
                                          T* Bt0, T* Bt1, f32x4 (&acc)[MT][NT]) {
  constexpr int PD = 3;  // chunks of A in flight
  constexpr int KC = Mma<T>::KC;
  constexpr int NS = KC / Mma<T>::KSTEP;
  typedef typename Mma<T>::Frag Frag;
  Pipe<T, MT, NT, PD> p;
  p.A = A; p.lda = lda; p.W = W; p.ldw = ldw; p.M = M; p.N = N; p.K = K; p.row0 = row0; p.n0 = n0;
  p.vec_ok = ((ldw * (int64_t)sizeof(T)) % 16 == 0) && ((uintptr_t)W % 16 == 0);
  p.nchunks = (int)((K + KC - 1) / KC);
  p.Bt0 = Bt0;
  p.Bt1 = Bt1;
  Frag a0[NS][MT], a1[NS][MT], a2[NS][MT];
  p.bs.load(W, ldw, K, N, 0, n0, p.vec_ok);
  load_a_chunk<T, MT>(A, lda, M, K, row0, 0, a0);
  if (p.nchunks > 1) load_a_chunk<T, MT>(A, lda, M, K, row0, KC, a1);
  if (p.nchunks > 2) load_a_chunk<T, MT>(A, lda, M, K, row0, 2 * KC, a2);
  __syncthreads();  // the LDS tiles may still be read by a previous phase
  p.bs.store(Bt0);
  __syncthreads();
  for (int ci = 0; ci < p.nchunks; ci += PD) {
    p.step(ci, a0, acc);
    if (ci + 1 < p.nchunks) p.step(ci + 1, a1, acc);
    if (ci + 2 < p.nchunks) p.step(ci + 2, a2, acc);
  }
}

// PLAIN / CONCAT
template <typename T, int MT, int NT>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmArgs g) {
  constexpr int LDB = Mma<T>::KC + Mma<T>::PAD;
  __shared__ __attribute__((aligned(16))) T Bt[2][NT * 16 * LDB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * (4 * MT * 16) + wave * MT * 16;
  const int64_t n0 = (int64_t)blockIdx.y * NT * 16;
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  mma_phase<T, MT, NT>(static_cast<const T*>(g.a), g.lda, static_cast<const T*>(g.w), g.ldw, g.M,
                       g.N, g.K, row0, n0, Bt[0], Bt[1], acc);
  if (g.mode == SAGA_GEMM_CONCAT)
    mma_phase<T, MT, NT>(static_cast<const T*>(g.a2), g.lda2, static_cast<const T*>(g.w2), g.ldw2,
                         g.M, g.N, g.K2, row0, n0, Bt[0], Bt[1], acc);
  // epilogue: lane holds rows 4*(lane/16) + r, column lane % 16 of each tile
  T* out = static_cast<T*>(g.out);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = row0 + mt * 16 + 4 * (lane >> 4) + r;
      if (row >= g.M) continue;
      const float rs = g.row_scale_deg ? rsqrt_deg(g.row_scale_deg[row]) : 1.0f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int64_t c = n0 + nt * 16 + (lane & 15);
        if (c >= g.N) continue;
        float v = acc[mt][nt][r] * rs;
        if (g.bias) v += g.bias[c];
        out[row * g.ldo + c] = Mma<T>::from_f(apply_act(g.act, v));
      }
    }
}

// GRU: acc1 = a w (input gates), acc2 = a2 w2 (hidden gates), column blocks
// (r, z, n) of width F = NT3 * 16; hidden state h = a2
template <typename T, int NT3>
__global__ __launch_bounds__(kThreads) void k_gemm_gru(GemmArgs g) {
  constexpr int NT = 3 * NT3;
  constexpr int LDB = Mma<T>::KC + Mma<T>::PAD;
  __shared__ __attribute__((aligned(16))) T Bt[2][NT * 16 * LDB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * (4 * 16) + wave * 16;
  f32x4 acc1[1][NT], acc2[1][NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    acc1[0][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc2[0][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const T* a = static_cast<const T*>(g.a);
  const T* h = static_cast<const T*>(g.a2);
  mma_phase<T, 1, NT>(a, g.lda, static_cast<const T*>(g.w), g.ldw, g.M, g.N, g.K, row0, 0, Bt[0],
                      Bt[1], acc1);
  mma_phase<T, 1, NT>(h, g.lda2, static_cast<const T*>(g.w2), g.ldw2, g.M, g.N, g.K2, row0, 0,
                      Bt[0], Bt[1], acc2);
  const int F = NT3 * 16;
  T* out = static_cast<T*>(g.out);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t row = row0 + 4 * (lane >> 4) + r;
    if (row >= g.M) continue;
#pragma unroll
    for (int t = 0; t < NT3; ++t) {
      const int c = t * 16 + (lane & 15);
      const float bi_r = g.bias ? g.bias[c] : 0.f, bi_z = g.bias ? g.bias[F + c] : 0.f,
                  bi_n = g.bias ? g.bias[2 * F + c] : 0.f;
      const float bh_r = g.bias2 ? g.bias2[c] : 0.f, bh_z = g.bias2 ? g.bias2[F + c] : 0.f,
                  bh_n = g.bias2 ? g.bias2[2 * F + c] : 0.f;
      const float rr = sigmoidf_(acc1[0][t][r] + bi_r + acc2[0][t][r] + bh_r);
      const float zz = sigmoidf_(acc1[0][t + NT3][r] + bi_z + acc2[0][t + NT3][r] + bh_z);
      const float nn = tanhf(acc1[0][t + 2 * NT3][r] + bi_n + rr * (acc2[0][t + 2 * NT3][r] + bh_n));
      const float hp = Mma<T>::to_f(h[row * g.lda2 + c]);
      out[row * g.ldo + c] = Mma<T>::from_f((1.0f - zz) * nn + zz * hp);
    }
  }
}

template <typename T, int MT, int NT>
hipError_t launch_plain(const GemmArgs& g, hipStream_t st) {
  const int64_t bm = 4 * MT * 16;
  dim3 grid((unsigned)((g.M + bm - 1) / bm), (unsigned)((g.N + NT * 16 - 1) / (NT * 16)));
  hipLaunchKernelGGL((k_gemm<T, MT, NT>), grid, dim3(kThreads), 0, st, g);
  return hipGetLastError();
}

// rows per wave for N <= 128 (2 x 16 = 32 rows by default); the
// SAGA_GEMM_MT environment variable (1, 2 or 4) overrides it for tuning
int gemm_mt() {
  static int v = [] {
    const char* e = getenv("SAGA_GEMM_MT");
    int x = e ? atoi(e) : 2;
    return (x == 1 || x == 2 || x == 4) ? x : 2;
  }();
  return v;
}

template <typename T, int NT>
hipError_t launch_nt(const GemmArgs& g, hipStream_t st) {
  switch (gemm_mt()) {
    case 1: return launch_plain<T, 1, NT>(g, st);
    case 2: return launch_plain<T, 2, NT>(g, st);
    default: return launch_plain<T, 4, NT>(g, st);
  }
}

template <typename T>
hipError_t dispatch(const GemmArgs& g, hipStream_t st) {
  if (g.mode == SAGA_GEMM_GRU) {
    const int64_t F = g.N / 3;
    dim3 grid((unsigned)((g.M + 63) / 64));
    switch (F) {
      case 16: hipLaunchKernelGGL((k_gemm_gru<T, 1>), grid, dim3(kThreads), 0, st, g); break;
      case 32: hipLaunchKernelGGL((k_gemm_gru<T, 2>), grid, dim3(kThreads), 0, st, g); break;
      case 48: hipLaunchKernelGGL((k_gemm_gru<T, 3>), grid, dim3(kThreads), 0, st, g); break;
      case 64: hipLaunchKernelGGL((k_gemm_gru<T, 4>), grid, dim3(kThreads), 0, st, g); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int64_t nt = (g.N + 15) / 16;
  if (nt <= 1) return launch_nt<T, 1>(g, st);
  if (nt <= 2) return launch_nt<T, 2>(g, st);
  if (nt <= 3) return launch_nt<T, 3>(g, st);
  if (nt <= 4) return launch_nt<T, 4>(g, st);
  if (nt <= 5) return launch_nt<T, 5>(g, st);
  if (nt <= 8) return launch_nt<T, 8>(g, st);
  return launch_plain<T, 2, 16>(g, st);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, hipStream_t st) {
  if (g.M == 0) return hipSuccess;
  return g.dtype == SAGA_BF16 ? dispatch<uint16_t>(g, st) : dispatch<float>(g, st);
}

}  // namespace saga
