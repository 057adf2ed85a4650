// kernels_fcn.hip -- fully-connected path of the structured-derivatives NTK on gfx950.
//
// For a dense layer y = theta x the Jacobian dy/dtheta = I (kron) x^T is constant-block
// diagonal, so the smallest sub-array to keep is the layer input x itself, and the
// NTK summand of layer l collapses to (x1 . x2) * (df1/dy)(df2/dy)^T (Eq.
// mixed_product_example; Section 4.1).  The kernels here compute
//   * the forward pass keeping every layer input h_l and act'(z_l)       (k_dense_fwd)
//   * the O one-hot output cotangents pulled back through all layers at once,
//     G_{l-1} = (G_l W_l) * act'(z_{l-1}) with rows (n, o)               (k_dense_bwd)
//   * the layer-input Grams h1_l h2_l^T (+1 with a bias)                 (k_gram)
//   * the fused contraction: per output tile, sum over layers of
//     gram_l[n1,n2] * (G1_l G2_l^T)[(n1,o1),(n2,o2)] in registers, plus the readout
//     summand gram_L[n1,n2] delta_{o1 o2}, written as theta[n1][n2][o1][o2]  (k_ntk_fcn)
#include "gemm_core.hpp"
#include "launch.hpp"

namespace ntk {

using CfgBig = TileCfg<128, 128, 32, 64, 64>;   // 4 waves, 64x64 per wave
using CfgSmall = TileCfg<64, 64, 32, 32, 32>;   // 4 waves, 32x32 per wave

static inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

template <class Cfg, class LA, class LB>
static hipError_t set_smem(const void* fn) {
  constexpr int bytes = gemm_smem_bytes<Cfg, LA, LB>();
  if (bytes > 65536)
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  return hipSuccess;
}

static inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// ------------------------------------------------------------------------------ forward
// The pre-activation is accumulated in fp64 from the fp32 layer input and weights, then
// the activation's decision (ReLU sign) is taken on that value and h_{l+1} is stored in fp32.
template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_fwd(LoadKInner la, LoadKInner lb, const float* __restrict__ bias, int M, int N, int act,
            float* __restrict__ hn, float* __restrict__ dphi, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f64x4 acc[Cfg::FM16][Cfg::FN16];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, 0, la.K, smem, acc);
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, double v) {
    if (r < M && c < N) {
      const double z = v + (bias ? (double)bias[c] : 0.0);
      float h, d;
      if (act == 1) {
        h = z > 0.0 ? (float)z : 0.f;
        d = z > 0.0 ? 1.f : 0.f;
      } else {
        const float zf = (float)z;
        h = act_fwd(act, zf);
        d = act_deriv(act, zf);
      }
      hn[(long long)r * N + c] = h;
      dphi[(long long)r * N + c] = d;
    }
  });
}

template <class Cfg>
static hipError_t dense_fwd_cfg(hipStream_t s, const float* h, const float* W, const float* b, int M,
                                int N, int K, int act, float* hn, float* dphi) {
  LoadKInner la{h, M, K, K, aligned16(h) && K % 4 == 0};
  LoadKInner lb{W, N, K, K, aligned16(W) && K % 4 == 0};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(M, Cfg::BM);
  hipError_t e = set_smem<Cfg, LoadKInner, LoadKInner>((const void*)k_dense_fwd<Cfg>);
  if (e != hipSuccess) return e;
  k_dense_fwd<Cfg><<<dim3(tm * tn), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, LoadKInner, LoadKInner>(), s>>>(la, lb, b, M, N, act, hn, dphi, tn);
  return hipGetLastError();
}

hipError_t launch_dense_fwd(hipStream_t s, const float* h, const float* W, const float* b, int M,
                            int N, int K, int act, float* hn, float* dphi) {
  return dense_fwd_cfg<CfgSmall>(s, h, W, b, M, N, K, act, hn, dphi);
}

// ------------------------------------------------------------------------------ backward
template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_bwd(LoadKInner la, LoadKInner lb, const float* __restrict__ dphi, int R, int N, int O,
            float* __restrict__ out, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, 0, la.K, smem, acc);
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, float v) {
    if (r < R && c < N) out[(long long)r * N + c] = v * dphi[(long long)(r / O) * N + c];
  });
}

template <class Cfg>
static hipError_t dense_bwd_cfg(hipStream_t s, const float* G, const float* Wt, const float* dphi,
                                int R, int N, int K, int O, float* out) {
  LoadKInner la{G, R, K, K, aligned16(G) && K % 4 == 0};
  LoadKInner lb{Wt, N, K, K, aligned16(Wt) && K % 4 == 0};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(R, Cfg::BM);
  hipError_t e = set_smem<Cfg, LoadKInner, LoadKInner>((const void*)k_dense_bwd<Cfg>);
  if (e != hipSuccess) return e;
  k_dense_bwd<Cfg><<<dim3(tm * tn), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, LoadKInner, LoadKInner>(), s>>>(la, lb, dphi, R, N, O, out, tn);
  return hipGetLastError();
}

hipError_t launch_dense_bwd(hipStream_t s, const float* G, const float* Wt, const float* dphi,
                            int R, int N, int K, int O, float* out) {
  const long long big_tiles = (long long)cdiv(R, 128) * cdiv(N, 128);
  if (big_tiles >= 512) return dense_bwd_cfg<CfgBig>(s, G, Wt, dphi, R, N, K, O, out);
  return dense_bwd_cfg<CfgSmall>(s, G, Wt, dphi, R, N, K, O, out);
}

// ------------------------------------------------------------------------------ seed, transpose
__global__ void k_bwd_seed(const float* __restrict__ W, const float* __restrict__ dphi, int M,
                           int O, int C, float* __restrict__ G) {
  const long long total = (long long)M * O * C;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(i % C);
    const long long mo = i / C;
    const int o = (int)(mo % O);
    const long long m = mo / O;
    G[i] = W[(long long)o * C + c] * dphi[m * C + c];
  }
}

hipError_t launch_bwd_seed(hipStream_t s, const float* W, const float* dphi, int M, int O, int C,
                           float* G) {
  const long long total = (long long)M * O * C;
  const int blocks = (int)std::min<long long>((total + 255) / 256, 256 * 64);
  k_bwd_seed<<<dim3(blocks), dim3(256), 0, s>>>(W, dphi, M, O, C, G);
  return hipGetLastError();
}

__global__ void k_transpose(const float* __restrict__ W, int R, int C, float* __restrict__ Wt) {
  __shared__ float tile[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int j = ty; j < 32; j += 8) {
    const int r = r0 + j, c = c0 + tx;
    if (r < R && c < C) tile[j][tx] = W[(long long)r * C + c];
  }
  __syncthreads();
  for (int j = ty; j < 32; j += 8) {
    const int c = c0 + j, r = r0 + tx;
    if (r < R && c < C) Wt[(long long)c * R + r] = tile[tx][j];
  }
}

hipError_t launch_transpose(hipStream_t s, const float* W, int R, int C, float* Wt) {
  k_transpose<<<dim3(cdiv(C, 32), cdiv(R, 32)), dim3(256), 0, s>>>(W, R, C, Wt);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------ Grams
template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_gram(GramBatch g, int N1, int N2, int tiles_n) {
  extern __shared__ float smem[];
  const int z = blockIdx.y;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int K = g.K[z];
  const bool vec = (K % 4 == 0) && ((reinterpret_cast<uintptr_t>(g.h1[z]) & 15) == 0) &&
                   ((reinterpret_cast<uintptr_t>(g.h2[z]) & 15) == 0);
  LoadKInner la{g.h1[z], N1, K, K, vec};
  LoadKInner lb{g.h2[z], N2, K, K, vec};
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, 0, K, smem, acc);
  float* out = g.out[z];
  const float beta = g.beta[z];
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, float v) {
    if (r < N1 && c < N2) out[(long long)r * N2 + c] = v + beta;
  });
}

hipError_t launch_gram(hipStream_t s, const GramBatch& g, int N1, int N2) {
  using Cfg = CfgSmall;
  const int tn = cdiv(N2, Cfg::BN), tm = cdiv(N1, Cfg::BM);
  hipError_t e = set_smem<Cfg, LoadKInner, LoadKInner>((const void*)k_gram<Cfg>);
  if (e != hipSuccess) return e;
  k_gram<Cfg><<<dim3(tm * tn, g.count), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, LoadKInner, LoadKInner>(), s>>>(g, N1, N2, tn);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------ fused contraction
// Tile index -> (tm, tn).  Symmetric: enumerate the upper triangle tm <= tn row by row.
__device__ __forceinline__ void tri_index(int t, int nt, int& tm, int& tn) {
  int r = 0, base = 0;
  while (base + (nt - r) <= t) {
    base += nt - r;
    ++r;
  }
  tm = r;
  tn = r + (t - base);
}

template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_ntk_fcn(FcnContraction c, int N1, int N2, int O, int symmetric, float* __restrict__ theta,
          int tiles_m, int tiles_n) {
  extern __shared__ float smem[];
  int tm, tn;
  if (symmetric) {
    tri_index(blockIdx.x, tiles_n, tm, tn);
  } else {
    tm = blockIdx.x / tiles_n;
    tn = blockIdx.x % tiles_n;
  }
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int R1 = N1 * O, R2 = N2 * O;

  f32x16 tot[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(tot);
  for (int l = 0; l < c.L; ++l) {
    const int K = c.K[l];
    const bool vec = (K % 4 == 0) && ((reinterpret_cast<uintptr_t>(c.G1[l]) & 15) == 0) &&
                     ((reinterpret_cast<uintptr_t>(c.G2[l]) & 15) == 0);
    LoadKInner la{c.G1[l], R1, K, K, vec};
    LoadKInner lb{c.G2[l], R2, K, K, vec};
    f32x16 acc[Cfg::FM][Cfg::FN];
    zero_acc<Cfg>(acc);
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, K, smem, acc);
    const float* gram = c.gram[l];
    // tot += gram_l[n1, n2] * acc   (the scalar x1.x2 of Eq. mixed_product_example)
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM, wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn) {
      const int s = n0 + wn0 + fn * 32 + (lane & 31);
      const int n2 = s < R2 ? s / O : 0;
#pragma unroll
      for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = m0 + wm0 + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
          const int n1 = r < R1 ? r / O : 0;
          tot[fm][fn][v] += gram[(long long)n1 * N2 + n2] * acc[fm][fn][v];
        }
    }
  }
  const float* gro = c.gram_readout;
  const bool mirror = symmetric && tm != tn;
  for_each_acc<Cfg>(tot, m0, n0, [&](int r, int s, float v) {
    if (r < R1 && s < R2) {
      const int n1 = r / O, o1 = r - n1 * O;
      const int n2 = s / O, o2 = s - n2 * O;
      if (o1 == o2) v += gro[(long long)n1 * N2 + n2];
      theta[(((long long)n1 * N2 + n2) * O + o1) * O + o2] = v;
      if (mirror) theta[(((long long)n2 * N1 + n1) * O + o2) * O + o1] = v;
    }
  });
}

hipError_t launch_ntk_fcn(hipStream_t s, const FcnContraction& c, int N1, int N2, int O,
                          int symmetric, float* theta) {
  const int R1 = N1 * O, R2 = N2 * O;
  auto go = [&](auto cfg_tag) -> hipError_t {
    using Cfg = decltype(cfg_tag);
    const int tm = cdiv(R1, Cfg::BM), tn = cdiv(R2, Cfg::BN);
    const int tiles = symmetric ? tn * (tn + 1) / 2 : tm * tn;
    hipError_t e = set_smem<Cfg, LoadKInner, LoadKInner>((const void*)k_ntk_fcn<Cfg>);
    if (e != hipSuccess) return e;
    k_ntk_fcn<Cfg><<<dim3(tiles), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, LoadKInner, LoadKInner>(), s>>>(c, N1, N2, O, symmetric, theta, tm, tn);
    return hipGetLastError();
  };
  const long long big_tiles = (long long)cdiv(R1, 128) * cdiv(R2, 128);
  if (big_tiles >= 512) return go(CfgBig{});
  return go(CfgSmall{});
}

}  // namespace ntk
