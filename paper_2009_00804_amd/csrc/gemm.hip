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

// stage rows [k0, k0 + KC) of W (columns [n0, n0 + NT*16)) transposed:
// Bt[n][k - k0]
template <typename T, int NT>
__device__ __forceinline__ void stage_b(const T* __restrict__ W, int64_t ldw, int64_t K,
                                        int64_t N, int64_t k0, int64_t n0, T* Bt) {
  constexpr int KC = Mma<T>::KC;
  constexpr int LDB = KC + Mma<T>::PAD;
  constexpr int BN = NT * 16;
  for (int idx = threadIdx.x; idx < KC * BN; idx += kThreads) {
    const int kk = idx / BN, nn = idx % BN;
    const int64_t k = k0 + kk, n = n0 + nn;
    T v = T(0);
    if (k < K && n < N) v = W[k * ldw + n];
    Bt[nn * LDB + kk] = v;
  }
}

template <typename T, int MT, int NT>
__device__ __forceinline__ void mma_phase(const T* __restrict__ A, int64_t lda, const T* __restrict__ W,
                                          int64_t ldw, int64_t M, int64_t N, int64_t K,
                                          int64_t row0, int64_t n0, T* Bt, f32x4 (&acc)[MT][NT]) {
  constexpr int EPL = Mma<T>::EPL;
  constexpr int KSTEP = Mma<T>::KSTEP;
  constexpr int KC = Mma<T>::KC;
  constexpr int LDB = KC + Mma<T>::PAD;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lg = lane >> 4;
  for (int64_t k0 = 0; k0 < K; k0 += KC) {
    __syncthreads();
    stage_b<T, NT>(W, ldw, K, N, k0, n0, Bt);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KC; kk += KSTEP) {
      if (k0 + kk >= K) break;
      typename Mma<T>::Frag af[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        af[mt] = load_a<T>(A, lda, row0 + mt * 16 + lr, k0 + kk + lg * EPL, M, K);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        typename Mma<T>::Frag bf;
        __builtin_memcpy(&bf, Bt + (nt * 16 + lr) * LDB + kk + lg * EPL, 16);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) Mma<T>::mma(af[mt], bf, acc[mt][nt]);
      }
    }
  }
}

// PLAIN / CONCAT
template <typename T, int MT, int NT>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmArgs g) {
  constexpr int LDB = Mma<T>::KC + Mma<T>::PAD;
  __shared__ __attribute__((aligned(16))) T Bt[NT * 16 * LDB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * (4 * MT * 16) + wave * MT * 16;
  const int64_t n0 = (int64_t)blockIdx.y * NT * 16;
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  mma_phase<T, MT, NT>(static_cast<const T*>(g.a), g.lda, static_cast<const T*>(g.w), g.ldw, g.M,
                       g.N, g.K, row0, n0, Bt, acc);
  if (g.mode == SAGA_GEMM_CONCAT)
    mma_phase<T, MT, NT>(static_cast<const T*>(g.a2), g.lda2, static_cast<const T*>(g.w2), g.ldw2,
                         g.M, g.N, g.K2, row0, n0, Bt, acc);
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
  __shared__ __attribute__((aligned(16))) T Bt[NT * 16 * LDB];
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
  mma_phase<T, 1, NT>(a, g.lda, static_cast<const T*>(g.w), g.ldw, g.M, g.N, g.K, row0, 0, Bt,
                      acc1);
  mma_phase<T, 1, NT>(h, g.lda2, static_cast<const T*>(g.w2), g.ldw2, g.M, g.N, g.K2, row0, 0, Bt,
                      acc2);
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
  if (nt <= 1) return launch_plain<T, 2, 1>(g, st);
  if (nt <= 2) return launch_plain<T, 2, 2>(g, st);
  if (nt <= 3) return launch_plain<T, 2, 3>(g, st);
  if (nt <= 4) return launch_plain<T, 2, 4>(g, st);
  if (nt <= 5) return launch_plain<T, 2, 5>(g, st);
  if (nt <= 8) return launch_plain<T, 2, 8>(g, st);
  return launch_plain<T, 1, 16>(g, st);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, hipStream_t st) {
  if (g.M == 0) return hipSuccess;
  return g.dtype == SAGA_BF16 ? dispatch<uint16_t>(g, st) : dispatch<float>(g, st);
}

}  // namespace saga
