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
#include <type_traits>

#include "gemm_core.hpp"
#include "launch.hpp"

namespace ntk {

using CfgBig = TileCfg<128, 128, 32, 64, 64>;   // 4 waves, 64x64 per wave
using CfgBig8 = TileCfg<128, 128, 32, 32, 64>;  // 8 waves, 32x64 per wave
using CfgSK = CfgBig8;                          // stream-K contraction
// The stream-K contraction keeps two workgroups per compute unit (two LDS stages each, so
// both fit the 160 KB of LDS): one workgroup's barrier waits are covered by the other's MFMAs.
constexpr int kSkPerCu = 2, kSkStages = 2;
// LDS stages of the direct-to-LDS loop of the layer-split contraction (64 x 64 tiles): two
// stages (32 KB) let four workgroups share a compute unit
constexpr int kSplitStages = 2;
// LDS stages of the Grams' direct-to-LDS loop (64 x 64 tiles)
constexpr int kGramStages = 3;
// the forward splits K (up to kFwdMaxSplits ways) below kFwdSplitTiles output tiles
constexpr int kFwdSplitTiles = 256, kFwdMaxSplits = 8;
using CfgSmall = TileCfg<64, 64, 32, 32, 32>;   // 4 waves, 32x32 per wave
using CfgPw = TileCfg<128, 64, 32, 32, 32>;     // pointwise backward, <= 64 channels: 8 waves
using CfgFwd64 = TileCfg<64, 64, 32, 32, 16>;   // fp64 forward: 8 waves, 32x16 per wave
using TrueT = std::true_type;
using FalseT = std::false_type;

static inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

template <class Cfg, class LA, class LB>
static hipError_t set_smem(const void* fn) {
  constexpr int bytes = gemm_smem_bytes<Cfg, LA, LB>();
  if (bytes > 65536)
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  return hipSuccess;
}

// ------------------------------------------------------------------------------ forward
// The pre-activation is accumulated in fp64 from the fp32 layer input and weights, then
// the activation's decision (ReLU sign) is taken on that value and h_{l+1} is stored in fp32.
__device__ __forceinline__ void fwd_epilogue(double z, int act, float& h, float& d) {
  if (act == 1) {
    h = z > 0.0 ? (float)z : 0.f;
    d = z > 0.0 ? 1.f : 0.f;
  } else {
    const float zf = (float)z;
    h = act_fwd(act, zf);
    d = act_deriv(act, zf);
  }
}

// With SEED (the last hidden layer), the epilogue also writes the readout cotangents
// sg[r, o, c] = sw[o, c] act'(z[r, c]) for o < so.
template <class Cfg, bool VEC, bool DMA, bool SEED = false>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_fwd(LoadKInnerT<VEC> la, LoadKInnerT<VEC> lb, const float* __restrict__ bias, int M, int N,
            int act, float* __restrict__ hn, float* __restrict__ dphi, int tiles_n,
            const float* __restrict__ sw = nullptr, int so = 0, float* __restrict__ sg = nullptr) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f64x4 acc[Cfg::FM16][Cfg::FN16];
  zero_acc<Cfg>(acc);
  if (DMA)
    gemm_mainloop_dma<Cfg, 3>(la.p, la.ld, la.rows, lb.p, lb.ld, lb.rows, m0, n0, 0, la.K, smem, acc);
  else
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, la.K, smem, acc);
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, double v) {
    const double b = bias ? (double)bias[min(c, N - 1)] : 0.0;
    float h, d;
    fwd_epilogue(v + b, act, h, d);
    if (r < M && c < N) {
      hn[(long long)r * N + c] = h;
      dphi[(long long)r * N + c] = d;
      if (SEED) {
        float* g = sg + (long long)r * so * N + c;
        for (int o = 0; o < so; ++o) g[(long long)o * N] = sw[(long long)o * N + c] * d;
      }
    }
  });
}

// Split-K form for a small batch (few output tiles): workgroup (tile, z) accumulates the K
// range [z chunk, (z+1) chunk) in fp64 and stores it; k_dense_fwd_reduce adds the partials in
// order, in fp64, and takes the activation's decision on that sum.
template <class Cfg, bool VEC, bool DMA>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_fwd_part(LoadKInnerT<VEC> la, LoadKInnerT<VEC> lb, int M, int N, int chunk,
                 double* __restrict__ part, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n, z = blockIdx.y;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int k0 = z * chunk, k1 = min(la.K, k0 + chunk);
  f64x4 acc[Cfg::FM16][Cfg::FN16];
  zero_acc<Cfg>(acc);
  if (DMA)
    gemm_mainloop_dma<Cfg, 3>(la.p, la.ld, la.rows, lb.p, lb.ld, lb.rows, m0, n0, k0, k1, smem, acc);
  else
    gemm_mainloop<Cfg>(la, lb, m0, n0, k0, k1, smem, acc);
  double* P = part + (long long)z * M * N;
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, double v) {
    if (r < M && c < N) P[(long long)r * N + c] = v;
  });
}

__global__ void __launch_bounds__(256)
k_dense_fwd_reduce(const double* __restrict__ part, int splits, int M, int N, const float* __restrict__ bias,
                   int act, float* __restrict__ hn, float* __restrict__ dphi, const float* __restrict__ sw,
                   int so, float* __restrict__ sg) {
  const long long total = (long long)M * N;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    double z = 0.0;
    for (int q = 0; q < splits; ++q) z += part[(long long)q * total + i];
    if (bias) z += (double)bias[i % N];
    float h, d;
    fwd_epilogue(z, act, h, d);
    hn[i] = h;
    dphi[i] = d;
    if (sg) {   // the readout cotangents of the last hidden layer
      const long long r = i / N, c = i - r * N;
      for (int o = 0; o < so; ++o) sg[(r * so + o) * N + c] = sw[(long long)o * N + c] * d;
    }
  }
}

// Block coordinates of the small-batch kernels: the tm x tn blocks of B x B outputs are numbered
// row by row (or column by column when by_cols) and cut into 8 contiguous ranges, one per XCD, so
// that an XCD reads a slice of the larger operand through its L2 (and all of the smaller one).
// False for the padding workgroups past an XCD's range.
__device__ __forceinline__ bool small_block_coords(int tiles_m, int tiles_n, int by_cols, int B, int& m0,
                                                   int& n0) {
  int blk;
  if (!xcd_block(blockIdx.x, tiles_m * tiles_n, blk)) return false;
  const int tm = by_cols ? blk % tiles_m : blk / tiles_n;
  const int tn = by_cols ? blk / tiles_m : blk % tiles_n;
  m0 = tm * B;
  n0 = tn * B;
  return true;
}

// Few rows and columns (a small batch): one 16 x 16 block of z per workgroup, so that even a
// 128 x 512 layer makes 256 workgroups without partial sums in memory.  The WAVES waves take
// every WAVES-th 16-column slice of K with the 16x16x4 fp64 MFMA on the exactly widened fp32
// values, and their partial blocks are added in wave order, in fp64, through LDS before the bias
// and the activation's decision (with sg, the last hidden layer also writes the readout
// cotangents).  A lane loads the four columns k0 + 4 (l / 16) + q (q = 0..3) of row l % 16 of
// both operands, and MFMA q contracts element q (the same column permutation for both
// operands); the fp64 MFMA returns D[4 v + l / 16][l % 16] in element v of lane l.
constexpr int kFwdSmallBlocks = 1024;   // at most this many 16 x 16 blocks (four per CU)
constexpr int kFwdSmallWaves = 8;
constexpr int kSeedPre = 16;
template <bool VEC, int WAVES>
__global__ void __launch_bounds__(64 * WAVES)
k_dense_fwd_small(const float* __restrict__ h, const float* __restrict__ W, const float* __restrict__ bias,
                  int M, int N, int K, int act, float* __restrict__ hn, float* __restrict__ dphi,
                  int tiles_m, int tiles_n, int by_cols, const float* __restrict__ sw, int so,
                  float* __restrict__ sg) {
  __shared__ double red[WAVES][256];
  int m0, n0;
  if (!small_block_coords(tiles_m, tiles_n, by_cols, 16, m0, n0)) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, kq = 4 * (lane >> 4);
  const bool va = m0 + i < M, vb = n0 + i < N;
  const float* __restrict__ pa = h + (long long)min(m0 + i, M - 1) * K;
  const float* __restrict__ pb = W + (long long)min(n0 + i, N - 1) * K;
  // the readout weights of this thread's output column for the fused seed, loaded ahead of
  // the K loop (up to kSeedPre outputs; more are read in the epilogue)
  const int r = m0 + (threadIdx.x >> 4), c = n0 + (threadIdx.x & 15);
  float swv[kSeedPre];
  if (sg && threadIdx.x < 256 && c < N) {
#pragma unroll
    for (int o = 0; o < kSeedPre; ++o) swv[o] = o < so ? sw[(long long)o * N + c] : 0.f;
  }
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  // batches of U slices: every load of a batch is issued before its MFMAs, from addresses
  // clamped into the rows (a column past K reads a valid element and is zeroed), so that the
  // loop body has no branch
  constexpr int U = 4;
  for (int kb = 16 * wave; kb < K; kb += 16 * WAVES * U) {
    f32x4 a[U], b[U];
    bool in[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kb + 16 * WAVES * u + kq;
      if (VEC) {   // K % 4 == 0 and 16-byte aligned rows: the 4 columns are all in or all out
        in[u] = k < K;
        const int kc = min(k, K - 4);
        a[u] = *reinterpret_cast<const f32x4*>(pa + kc);
        b[u] = *reinterpret_cast<const f32x4*>(pb + kc);
      } else {
        in[u] = true;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int kc = min(k + q, K - 1);
          const float x = pa[kc], y = pb[kc];
          a[u][q] = k + q < K ? x : 0.f;
          b[u][q] = k + q < K ? y : 0.f;
        }
      }
    }
    // keep the loads of the batch ahead of its MFMAs
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool use_a = va && in[u], use_b = vb && in[u];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(use_a ? (double)a[u][q] : 0.0, use_b ? (double)b[u][q] : 0.0,
                                                   acc, 0, 0, 0);
    }
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) red[wave][(4 * v + (lane >> 4)) * 16 + i] = acc[v];
  __syncthreads();
  if (threadIdx.x < 256 && r < M && c < N) {
    double z = red[0][threadIdx.x];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) z += red[w][threadIdx.x];
    if (bias) z += (double)bias[c];
    float hv, dv;
    fwd_epilogue(z, act, hv, dv);
    hn[(long long)r * N + c] = hv;
    dphi[(long long)r * N + c] = dv;
    // the readout cotangents of the last hidden layer, G[r, o, c] = Wr[o, c] act'(z[r, c])
    if (sg) {
      float* g = sg + (long long)r * so * N + c;
#pragma unroll
      for (int o = 0; o < kSeedPre; ++o)
        if (o < so) g[(long long)o * N] = swv[o] * dv;
      for (int o = kSeedPre; o < so; ++o) g[(long long)o * N] = sw[(long long)o * N + c] * dv;
    }
  }
}

bool dense_fwd_small_ok(long long M, long long N) {
  return M > 0 && N > 0 && (long long)cdiv(M, 64) * cdiv(N, 64) < kFwdSplitTiles &&
         (long long)cdiv(M, 16) * cdiv(N, 16) <= kFwdSmallBlocks;
}

long long dense_fwd_part_doubles(long long max_rows, long long max_cols) {
  // the split form only runs below kFwdSplitTiles output tiles of 64 x 64
  return std::min<long long>(kFwdMaxSplits * max_rows * max_cols,
                             (long long)kFwdMaxSplits * kFwdSplitTiles * 64 * 64);
}

template <class Cfg, bool VEC, bool DMA = false>
static hipError_t dense_fwd_cfg(hipStream_t s, const float* h, const float* W, const float* b, int M,
                                int N, int K, int act, float* hn, float* dphi, double* part,
                                long long part_capacity, const float* sw, int so, float* sg) {
  using L = LoadKInnerT<VEC>;
  L la{h, M, K, K};
  L lb{W, N, K, K};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(M, Cfg::BM);
  constexpr int bytes = DMA ? gemm_dma_smem_bytes<Cfg, 3>() : gemm_smem_bytes<Cfg, L, L>();
  // split K when the tiles alone would leave most compute units idle
  int splits = 1, chunk = K;
  if (part && tm * tn < kFwdSplitTiles) {
    const int want = std::min<int>(kFwdMaxSplits, cdiv(2 * kFwdSplitTiles, tm * tn));
    chunk = std::max(2 * Cfg::BK, cdiv(cdiv(K, want), Cfg::BK) * Cfg::BK);
    splits = cdiv(K, chunk);
    if ((long long)splits * M * N > part_capacity) splits = 1;
  }
  if (splits > 1) {
    hipError_t e = hipFuncSetAttribute((const void*)k_dense_fwd_part<Cfg, VEC, DMA>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    k_dense_fwd_part<Cfg, VEC, DMA><<<dim3(tm * tn, splits), dim3(Cfg::THREADS), bytes, s>>>(
        la, lb, M, N, chunk, part, tn);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long long total = (long long)M * N;
    k_dense_fwd_reduce<<<dim3((unsigned)std::min<long long>((total + 255) / 256, 4096)), dim3(256), 0, s>>>(
        part, splits, M, N, b, act, hn, dphi, sw, so, sg);
    return hipGetLastError();
  }
  auto go = [&](auto kern) -> hipError_t {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    kern<<<dim3(tm * tn), dim3(Cfg::THREADS), bytes, s>>>(la, lb, b, M, N, act, hn, dphi, tn, sw, so, sg);
    return hipGetLastError();
  };
  return sg ? go(k_dense_fwd<Cfg, VEC, DMA, true>) : go(k_dense_fwd<Cfg, VEC, DMA, false>);
}

hipError_t launch_dense_fwd(hipStream_t s, const float* h, const float* W, const float* b, int M,
                            int N, int K, int act, float* hn, float* dphi, double* part,
                            long long part_capacity, const float* seedW, int seedO, float* seedG) {
  const bool v = vec_ok(h, K, K) && vec_ok(W, K, K);
  if (M <= 0 || N <= 0) return hipSuccess;
  if (dense_fwd_small_ok(M, N)) {
    const long long blocks16 = (long long)cdiv(M, 16) * cdiv(N, 16);
    const int tm = cdiv(M, 16), tn = cdiv(N, 16);
    const int by_cols = M < N;   // each XCD reads a slice of the larger operand
    const dim3 grid((unsigned)(8 * cdiv(blocks16, 8)));
    constexpr int WV = kFwdSmallWaves;
    if (v)
      k_dense_fwd_small<true, WV><<<grid, dim3(64 * WV), 0, s>>>(h, W, b, M, N, K, act, hn, dphi, tm, tn, by_cols,
                                                                 seedW, seedO, seedG);
    else
      k_dense_fwd_small<false, WV><<<grid, dim3(64 * WV), 0, s>>>(h, W, b, M, N, K, act, hn, dphi, tm, tn, by_cols,
                                                                  seedW, seedO, seedG);
    return hipGetLastError();
  }
  if (v && K % 32 == 0 && dma_span_ok(K, K, 256))
    return dense_fwd_cfg<CfgFwd64, true, true>(s, h, W, b, M, N, K, act, hn, dphi, part, part_capacity, seedW,
                                               seedO, seedG);
  if (v)
    return dense_fwd_cfg<CfgFwd64, true>(s, h, W, b, M, N, K, act, hn, dphi, part, part_capacity, seedW, seedO,
                                         seedG);
  return dense_fwd_cfg<CfgFwd64, false>(s, h, W, b, M, N, K, act, hn, dphi, part, part_capacity, seedW, seedO,
                                        seedG);
}

// ------------------------------------------------------------------------------ backward
// out[r, c] = acc[r, c] * dphi[r / O, c]
struct EpiBwd {
  const float* dphi;
  float* out;
  int R, N;
  FastDiv fO;
  // Per 32-row MFMA fragment inside R: the out rows and the dphi rows r / O are addressed from
  // two wave-uniform bases (rows r0 and r0 / O) with 32-bit byte offsets (N < 2^25), and the 16
  // row quotients of a lane are shared by its column fragments.
  template <class Cfg>
  __device__ __forceinline__ void tile(f32x16 (&acc)[Cfg::FM][Cfg::FN], int m0, int n0) const {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
    const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
#pragma unroll
    for (int fm = 0; fm < Cfg::FM; ++fm) {
      const int r0 = __builtin_amdgcn_readfirstlane(m0 + wm0 + fm * 32);
      if (r0 >= R) continue;
      if (r0 + 32 <= R && N < (1 << 25)) {
        const int q0 = (int)fO.div(r0);
        float* ob = out + (long long)r0 * N;
        const float* db = dphi + (long long)q0 * N;
        int dq[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int i = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
          dq[v] = ((int)fO.div(r0 + i) - q0) * N;
        }
#pragma unroll
        for (int fn = 0; fn < Cfg::FN; ++fn) {
          const int c = n0 + wn0 + fn * 32 + (lane & 31);
          if (c >= N) continue;
          float d[16];
#pragma unroll
          for (int v = 0; v < 16; ++v) d[v] = at_bytes(db, (uint32_t)(dq[v] + c) * 4u);
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int i = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
            at_bytes(ob, (uint32_t)(i * N + c) * 4u) = acc[fm][fn][v] * d[v];
          }
        }
      } else {
#pragma unroll
        for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int r = r0 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
            const int c = n0 + wn0 + fn * 32 + (lane & 31);
            if (r < R && c < N) out[(long long)r * N + c] = acc[fm][fn][v] * dphi[(long long)fO.div(r) * N + c];
          }
      }
    }
  }
  __device__ __forceinline__ void elem(int r, int c, float v) const {
    if (r < R && c < N) out[(long long)r * N + c] = v * dphi[(long long)fO.div(r) * N + c];
  }
};

// Pointwise-convolution form: rows r = (img*O + o)*D + p of cotangent pixels; the act' of the
// layer before is per image pixel, dphi[img*D + p, c] (null: the identity).
struct EpiBwdPix {
  const float* dphi;
  float* out;
  int R, N;
  FastDiv fOD, fD;
  template <class Cfg>
  __device__ __forceinline__ void tile(f32x16 (&acc)[Cfg::FM][Cfg::FN], int m0, int n0) const {
    store_pixel_rows<Cfg>(acc, m0, n0, dphi, out, R, N, fOD, fD);
  }
};

template <class Cfg, bool VEC, bool DMA, class Epi = EpiBwd>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_bwd(LoadKInnerT<VEC> la, LoadKInnerT<VEC> lb, Epi epi, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  if (DMA)
    gemm_mainloop_dma<Cfg, 2>(la.p, la.ld, la.rows, lb.p, lb.ld, lb.rows, m0, n0, 0, la.K, smem, acc);
  else
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, la.K, smem, acc);
  epi.template tile<Cfg>(acc, m0, n0);
}

template <class Cfg, bool VEC, bool DMA = false>
static hipError_t dense_bwd_cfg(hipStream_t s, const float* G, const float* Wt, const float* dphi,
                                int R, int N, int K, int O, float* out) {
  using L = LoadKInnerT<VEC>;
  L la{G, R, K, K};
  L lb{Wt, N, K, K};
  EpiBwd epi{dphi, out, R, N, FastDiv((uint32_t)O)};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(R, Cfg::BM);
  constexpr int bytes = DMA ? gemm_dma_smem_bytes<Cfg, 2>() : gemm_smem_bytes<Cfg, L, L>();
  hipError_t e = hipFuncSetAttribute((const void*)k_dense_bwd<Cfg, VEC, DMA>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_dense_bwd<Cfg, VEC, DMA><<<dim3(tm * tn), dim3(Cfg::THREADS), bytes, s>>>(la, lb, epi, tn);
  return hipGetLastError();
}

// The same product with B read from W [K, N] itself (row k of W holds B[k][.]) through the
// K-outer tile layout, so that no transposed copy of W is needed.
template <class Cfg>
__device__ __forceinline__ void dense_bwd_ko_tile(const float* __restrict__ G, const float* __restrict__ W, int R,
                                                  int N, int K, const EpiBwd& epi, int tiles_n, int bx, float* smem) {
  const int tm = bx / tiles_n, tn = bx % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  DmaRowMajor<Cfg::BM, Cfg::WAVES> ia{G, K, R};
  DmaKOuterRowMajor<Cfg::BN, Cfg::WAVES> ib{W, N, N, K};
  gemm_mainloop_dma_ops<Cfg, 2>(ia, ib, m0, n0, 0, K, smem, acc);
  epi.template tile<Cfg>(acc, m0, n0);
}

template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_bwd_ko(const float* __restrict__ G, const float* __restrict__ W, int R, int N, int K, EpiBwd epi,
               int tiles_n) {
  extern __shared__ float smem[];
  dense_bwd_ko_tile<Cfg>(G, W, R, N, K, epi, tiles_n, blockIdx.x, smem);
}

// Few output tiles: each 64 x 64 tile by 8 waves in two groups of 4, group g taking half of the K
// tiles with LDS stages of its own (both halves the same number of K tiles, so that the groups
// meet at every barrier of the loop; K % 64 == 0).  Group 1 hands its partial tile to group 0
// through LDS, which adds it to its own and runs the epilogue: per wave the MFMA chain is half as
// long, and two waves share each SIMD (depth-4 width-512 FCN: 41.7 -> 39.9 us for its three
// backward layers).
constexpr int kBwdKSplitStages = 2;
template <class Cfg>
__global__ void __launch_bounds__(2 * Cfg::THREADS)
k_dense_bwd_ko2(const float* __restrict__ G, const float* __restrict__ W, int R, int N, int K, EpiBwd epi,
                int tiles_n) {
  extern __shared__ float smem[];
  constexpr int GROUP_FLOATS = gemm_dma_smem_bytes<Cfg, kBwdKSplitStages>() / 4;
  static_assert(Cfg::FM * Cfg::FN * Cfg::WAVES * 64 * 16 <= GROUP_FLOATS, "partial tile fits the LDS");
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = __builtin_amdgcn_readfirstlane(wave / Cfg::WAVES), lw = wave - g * Cfg::WAVES;
  const int half = K / 64 * 32;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  DmaRowMajor<Cfg::BM, Cfg::WAVES> ia{G, K, R};
  DmaKOuterRowMajor<Cfg::BN, Cfg::WAVES> ib{W, N, N, K};
  gemm_mainloop_dma_ops_w<Cfg, kBwdKSplitStages>(ia, ib, m0, n0, g * half, g ? K : half, smem + g * GROUP_FLOATS,
                                                 acc, lw, lane);
  // the loop ended with a barrier: the stages are free for group 1's partial tile
  f32x16* xs = reinterpret_cast<f32x16*>(smem);
  if (g == 1) {
#pragma unroll
    for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < Cfg::FN; ++fn) xs[((fm * Cfg::FN + fn) * Cfg::WAVES + lw) * 64 + lane] = acc[fm][fn];
  }
  __syncthreads();
  if (g == 1) return;
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn) acc[fm][fn] += xs[((fm * Cfg::FN + fn) * Cfg::WAVES + lw) * 64 + lane];
  epi.template tile<Cfg>(acc, m0, n0);
}

template <class Cfg>
static hipError_t dense_bwd_ko2_cfg(hipStream_t s, const float* G, const float* W, const float* dphi, int R,
                                    int N, int K, int O, float* out) {
  EpiBwd epi{dphi, out, R, N, FastDiv((uint32_t)O)};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(R, Cfg::BM);
  constexpr int bytes = 2 * gemm_dma_smem_bytes<Cfg, kBwdKSplitStages>();
  hipError_t e = hipFuncSetAttribute((const void*)k_dense_bwd_ko2<Cfg>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_dense_bwd_ko2<Cfg><<<dim3(tm * tn), dim3(2 * Cfg::THREADS), bytes, s>>>(G, W, R, N, K, epi, tn);
  return hipGetLastError();
}

template <class Cfg>
static hipError_t dense_bwd_ko_cfg(hipStream_t s, const float* G, const float* W, const float* dphi, int R,
                                   int N, int K, int O, float* out) {
  EpiBwd epi{dphi, out, R, N, FastDiv((uint32_t)O)};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(R, Cfg::BM);
  constexpr int bytes = gemm_dma_smem_bytes<Cfg, 2>();
  hipError_t e = hipFuncSetAttribute((const void*)k_dense_bwd_ko<Cfg>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_dense_bwd_ko<Cfg><<<dim3(tm * tn), dim3(Cfg::THREADS), bytes, s>>>(G, W, R, N, K, epi, tn);
  return hipGetLastError();
}

template <class Cfg, bool VEC, bool DMA = false>
static hipError_t pw_bwd_cfg(hipStream_t s, const float* G, const float* Wt, const float* dphi, int R, int N,
                             int K, int O, int D, float* out) {
  using L = LoadKInnerT<VEC>;
  L la{G, R, K, K};
  L lb{Wt, N, K, K};
  EpiBwdPix epi{dphi, out, R, N, FastDiv((uint32_t)(O * D)), FastDiv((uint32_t)D)};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(R, Cfg::BM);
  constexpr int bytes = DMA ? gemm_dma_smem_bytes<Cfg, 2>() : gemm_smem_bytes<Cfg, L, L>();
  hipError_t e = hipFuncSetAttribute((const void*)k_dense_bwd<Cfg, VEC, DMA, EpiBwdPix>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_dense_bwd<Cfg, VEC, DMA, EpiBwdPix><<<dim3(tm * tn), dim3(Cfg::THREADS), bytes, s>>>(la, lb, epi, tn);
  return hipGetLastError();
}

hipError_t launch_pw_bwd(hipStream_t s, const float* G, const float* Wt, const float* dphi, int R, int N,
                         int K, int O, int D, float* out) {
  if ((long long)O * D >= (1LL << 31) || R <= 0) return R <= 0 ? hipSuccess : hipErrorInvalidValue;
  const long long big_tiles = (long long)cdiv(R, 128) * cdiv(N, 128);
  const bool v = vec_ok(G, K, K) && vec_ok(Wt, K, K);
  // at most 64 output channels: 128x64 tiles (8 waves of 32x32), no half-empty 128-wide tile; a
  // memory-bound product (K = input channels), so the tile is sized for three workgroups per CU
  // (48 KB of LDS): 150 vs 160 us for 256x64 tiles at 1280 x 32x32 cotangent images of 64 channels
  if (N <= 64 && (long long)cdiv(R, 256) >= 512 && v && K % 32 == 0 && dma_span_ok(K, K, 256))
    return pw_bwd_cfg<CfgPw, true, true>(s, G, Wt, dphi, R, N, K, O, D, out);
  if (big_tiles >= 512) {
    if (v && K % 32 == 0 && dma_span_ok(K, K, 256)) return pw_bwd_cfg<CfgBig8, true, true>(s, G, Wt, dphi, R, N, K, O, D, out);
    return v ? pw_bwd_cfg<CfgBig8, true>(s, G, Wt, dphi, R, N, K, O, D, out)
             : pw_bwd_cfg<CfgBig8, false>(s, G, Wt, dphi, R, N, K, O, D, out);
  }
  return v ? pw_bwd_cfg<CfgSmall, true>(s, G, Wt, dphi, R, N, K, O, D, out)
           : pw_bwd_cfg<CfgSmall, false>(s, G, Wt, dphi, R, N, K, O, D, out);
}

// Two 8-wave workgroups share a compute unit (4 waves per SIMD).  At the depth-8 width-2048
// shape 1280 tiles over 512 slots leave the last round half empty, but both alternatives that
// remove it measured slower: a full stream-K schedule at one workgroup per CU (113 vs 122
// TFLOP/s), and persistent data-parallel rounds with a stream-K tail split along K at two
// workgroups per CU (4.91 vs 4.61 ms for the 7 layers) -- the tail round runs one workgroup
// per CU, faster than a full round.
hipError_t launch_dense_bwd(hipStream_t s, const float* G, const float* Wt, const float* dphi,
                            int R, int N, int K, int O, float* out) {
  const long long big_tiles = (long long)cdiv(R, 128) * cdiv(N, 128);
  const bool v = vec_ok(G, K, K) && vec_ok(Wt, K, K);
  if (big_tiles >= 512) {
    if (v && K % 32 == 0 && dma_span_ok(K, K, 256)) return dense_bwd_cfg<CfgBig8, true, true>(s, G, Wt, dphi, R, N, K, O, out);
    return v ? dense_bwd_cfg<CfgBig8, true>(s, G, Wt, dphi, R, N, K, O, out)
             : dense_bwd_cfg<CfgBig8, false>(s, G, Wt, dphi, R, N, K, O, out);
  }
  if (v && K % 32 == 0 && dma_span_ok(K, K, 256)) return dense_bwd_cfg<CfgSmall, true, true>(s, G, Wt, dphi, R, N, K, O, out);
  return v ? dense_bwd_cfg<CfgSmall, true>(s, G, Wt, dphi, R, N, K, O, out)
           : dense_bwd_cfg<CfgSmall, false>(s, G, Wt, dphi, R, N, K, O, out);
}

bool dense_bwd_w_ok(const float* G, const float* W, long long R, long long N, long long K) {
  return R > 0 && R < (1LL << 31) && K % 32 == 0 && K > 0 && N % 4 == 0 && N >= 4 &&
         vec_ok(G, K, K) && vec_ok(W, N, N) && dma_span_ok(K, K, 256) && K * N * 4 < (1LL << 31);
}

hipError_t launch_dense_bwd_w(hipStream_t s, const float* G, const float* W, const float* dphi, int R, int N,
                              int K, int O, float* out) {
  if (O <= 0) return hipErrorInvalidValue;
  if (!dense_bwd_w_ok(G, W, R, N, K)) return hipErrorInvalidValue;
  const long long big_tiles = (long long)cdiv(R, 128) * cdiv(N, 128);
  if (big_tiles >= 512) return dense_bwd_ko_cfg<CfgBig8>(s, G, W, dphi, R, N, K, O, out);
  if (K % 64 == 0) return dense_bwd_ko2_cfg<CfgSmall>(s, G, W, dphi, R, N, K, O, out);
  return dense_bwd_ko_cfg<CfgSmall>(s, G, W, dphi, R, N, K, O, out);
}

// ------------------------------------------------------------------------------ transpose
// One 32 x 32 tile of Wt = W^T (W is R x C, row-major), staged through LDS.
__device__ __forceinline__ void transpose_tile(const float* __restrict__ W, int R, int C, float* __restrict__ Wt,
                                               int c0, int r0, float (*tile)[33]) {
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

// The same for R and C multiples of 4 with 16-byte aligned rows: a 64 x 64 tile, every global
// access a float4 (a row quad of W read, a column quad of W written as a row quad of Wt).
__device__ __forceinline__ void transpose_tile4(const float* __restrict__ W, int R, int C, float* __restrict__ Wt,
                                                int c0, int r0, float (*tile)[65]) {
  const int q = threadIdx.x & 15, rr = threadIdx.x >> 4;   // quad within a 64-wide row, row 0..15
#pragma unroll
  for (int j = 0; j < 64; j += 16) {
    const int r = r0 + rr + j, c = c0 + 4 * q;
    if (r < R && c < C) {
      const float4 v = *reinterpret_cast<const float4*>(W + (long long)r * C + c);
      tile[rr + j][4 * q] = v.x;
      tile[rr + j][4 * q + 1] = v.y;
      tile[rr + j][4 * q + 2] = v.z;
      tile[rr + j][4 * q + 3] = v.w;
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 64; j += 16) {
    const int c = c0 + rr + j, r = r0 + 4 * q;
    if (r < R && c < C) {
      const float4 v = {tile[4 * q][rr + j], tile[4 * q + 1][rr + j], tile[4 * q + 2][rr + j], tile[4 * q + 3][rr + j]};
      *reinterpret_cast<float4*>(Wt + (long long)c * R + r) = v;
    }
  }
}

__global__ void __launch_bounds__(256) k_transpose(const float* __restrict__ W, int R, int C, float* __restrict__ Wt) {
  __shared__ float tile[32][33];
  transpose_tile(W, R, C, Wt, blockIdx.x * 32, blockIdx.y * 32, tile);
}

__global__ void __launch_bounds__(256) k_transpose4(const float* __restrict__ W, int R, int C, float* __restrict__ Wt) {
  __shared__ float tile[64][65];
  transpose_tile4(W, R, C, Wt, blockIdx.x * 64, blockIdx.y * 64, tile);
}

// Several transposes in one launch: matrix z = blockIdx.z; workgroups past its tile grid exit.
template <bool VEC4>
__global__ void __launch_bounds__(256) k_transpose_batch(TransposeBatch b) {
  constexpr int T = VEC4 ? 64 : 32;
  __shared__ float tile[T][T + 1];
  const int z = blockIdx.z;
  const int R = b.R[z], C = b.C[z];
  const int c0 = blockIdx.x * T, r0 = blockIdx.y * T;
  if (c0 >= C || r0 >= R) return;
  if constexpr (VEC4)
    transpose_tile4(b.W[z], R, C, b.Wt[z], c0, r0, tile);
  else
    transpose_tile(b.W[z], R, C, b.Wt[z], c0, r0, tile);
}

hipError_t launch_transpose(hipStream_t s, const float* W, int R, int C, float* Wt) {
  if (R % 4 == 0 && C % 4 == 0 && vec_ok(W, C, C) && vec_ok(Wt, R, R)) {
    k_transpose4<<<dim3(cdiv(C, 64), cdiv(R, 64)), dim3(256), 0, s>>>(W, R, C, Wt);
    return hipGetLastError();
  }
  k_transpose<<<dim3(cdiv(C, 32), cdiv(R, 32)), dim3(256), 0, s>>>(W, R, C, Wt);
  return hipGetLastError();
}

hipError_t launch_transpose_batch(hipStream_t s, const TransposeBatch& b) {
  if (b.count <= 0) return hipSuccess;
  if (b.count > kMaxLayers) return hipErrorInvalidValue;
  bool v4 = true;
  int maxR = 0, maxC = 0;
  for (int z = 0; z < b.count; ++z) {
    v4 = v4 && b.R[z] % 4 == 0 && b.C[z] % 4 == 0 && vec_ok(b.W[z], b.C[z], b.C[z]) && vec_ok(b.Wt[z], b.R[z], b.R[z]);
    maxR = std::max(maxR, b.R[z]);
    maxC = std::max(maxC, b.C[z]);
  }
  if (v4)
    k_transpose_batch<true><<<dim3(cdiv(maxC, 64), cdiv(maxR, 64), b.count), dim3(256), 0, s>>>(b);
  else
    k_transpose_batch<false><<<dim3(cdiv(maxC, 32), cdiv(maxR, 32), b.count), dim3(256), 0, s>>>(b);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------ Grams
template <class Cfg, bool VEC, bool DMA>
__global__ void __launch_bounds__(Cfg::THREADS)
k_gram(GramBatch g, int N1, int N2, int tiles_n) {
  extern __shared__ float smem[];
  const int z = blockIdx.y;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int K = g.K[z];
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  if (DMA) {
    gemm_mainloop_dma<Cfg, kGramStages>(g.h1[z], K, N1, g.h2[z], K, N2, m0, n0, 0, K, smem, acc);
  } else {
    LoadKInnerT<VEC> la{g.h1[z], N1, K, K};
    LoadKInnerT<VEC> lb{g.h2[z], N2, K, K};
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, K, smem, acc);
  }
  float* out = g.out[z];
  const float beta = g.beta[z];
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, float v) {
    if (r < N1 && c < N2) out[(long long)r * N2 + c] = v + beta;
  });
}

template <bool VEC, bool DMA>
static hipError_t gram_vec(hipStream_t s, const GramBatch& g, int N1, int N2) {
  using Cfg = CfgSmall;
  using L = LoadKInnerT<VEC>;
  const int tn = cdiv(N2, Cfg::BN), tm = cdiv(N1, Cfg::BM);
  constexpr int bytes = DMA ? gemm_dma_smem_bytes<Cfg, kGramStages>() : gemm_smem_bytes<Cfg, L, L>();
  hipError_t e = hipFuncSetAttribute((const void*)k_gram<Cfg, VEC, DMA>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_gram<Cfg, VEC, DMA><<<dim3(tm * tn, g.count), dim3(Cfg::THREADS), bytes, s>>>(g, N1, N2, tn);
  return hipGetLastError();
}

// Strided batch of Grams: out[b][n1][n2] = a1[n1 ld + b bs : + K] . a2[n2 ld + b bs : + K] for
// b < batches (one 64 x 64 tile of batch blockIdx.y per workgroup).
template <class Cfg, bool VEC, bool DMA>
__global__ void __launch_bounds__(Cfg::THREADS)
k_gram_strided(const float* __restrict__ a1, const float* __restrict__ a2, int N1, int N2, int K, long long ld,
               long long bs, float* __restrict__ out, int tiles_n) {
  extern __shared__ float smem[];
  const int b = blockIdx.y;
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  if (DMA) {
    gemm_mainloop_dma<Cfg, kGramStages>(a1 + b * bs, ld, N1, a2 + b * bs, ld, N2, m0, n0, 0, K, smem, acc);
  } else {
    LoadKInnerT<VEC> la{a1 + b * bs, N1, K, ld};
    LoadKInnerT<VEC> lb{a2 + b * bs, N2, K, ld};
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, K, smem, acc);
  }
  float* o = out + (long long)b * N1 * N2;
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, float v) {
    if (r < N1 && c < N2) o[(long long)r * N2 + c] = v;
  });
}

hipError_t launch_gram_strided(hipStream_t s, const float* a1, const float* a2, int N1, int N2, int K,
                               long long ld, long long bs, int batches, float* out) {
  if (batches <= 0 || N1 <= 0 || N2 <= 0) return hipSuccess;
  if (batches > 65535) return hipErrorInvalidValue;
  using Cfg = CfgSmall;
  const int tn = cdiv(N2, Cfg::BN), tm = cdiv(N1, Cfg::BM);
  const bool v = vec_ok(a1, ld, K) && vec_ok(a2, ld, K) && bs % 4 == 0;
  const bool dma = v && K % 32 == 0 && dma_span_ok(ld, K, 256);
  auto go = [&](auto vec_tag, auto dma_tag) -> hipError_t {
    constexpr bool VEC = decltype(vec_tag)::value, DMA = decltype(dma_tag)::value;
    using L = LoadKInnerT<VEC>;
    constexpr int bytes = DMA ? gemm_dma_smem_bytes<Cfg, kGramStages>() : gemm_smem_bytes<Cfg, L, L>();
    hipError_t e = hipFuncSetAttribute((const void*)k_gram_strided<Cfg, VEC, DMA>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    k_gram_strided<Cfg, VEC, DMA><<<dim3(tm * tn, batches), dim3(Cfg::THREADS), bytes, s>>>(a1, a2, N1, N2, K, ld,
                                                                                          bs, out, tn);
    return hipGetLastError();
  };
  if (dma) return go(TrueT{}, TrueT{});
  return v ? go(TrueT{}, FalseT{}) : go(FalseT{}, FalseT{});
}

// Small batches: the 64 x 64 tiles of k_gram would leave most compute units idle, so workgroup
// (block, z) computes one 16 x 16 block of layer z's Gram with the 16x16x4 fp32 MFMA, its four
// waves taking every fourth 16-column slice of K; the waves' partial blocks are then added in
// wave order through LDS.  The MFMA takes A[i][k] from lane i + 16 k and B[k][j] from lane
// j + 16 k, and returns D[4 (l / 16) + v][l % 16] in register v of lane l.  Lane l loads the four
// columns k0 + 4 (l / 16) + q (q = 0..3) of row l % 16 of both operands, and MFMA q contracts
// element q of both, so the four MFMAs cover the 16 columns of the slice (in a permuted order,
// the same for both operands).
template <bool VEC>
__device__ __forceinline__ void gram_small_block(const GramBatch& g, int N1, int N2, int tiles_n, int bx, int z,
                                                 float (*red)[256]) {
  const int m0 = (bx / tiles_n) * 16, n0 = (bx % tiles_n) * 16;
  const int K = g.K[z];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = lane & 15, kq = 4 * (lane >> 4);
  const bool va = m0 + i < N1, vb = n0 + i < N2;
  const float* __restrict__ pa = g.h1[z] + (long long)min(m0 + i, N1 - 1) * K;
  const float* __restrict__ pb = g.h2[z] + (long long)min(n0 + i, N2 - 1) * K;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  // batches of U slices: every load of a batch is issued before its MFMAs, from addresses
  // clamped into the rows (a column past K reads a valid element and is zeroed), so that the
  // loop body has no branch
  constexpr int U = 4;
  for (int kb = 16 * wave; kb < K; kb += 64 * U) {
    f32x4 a[U], b[U];
    bool in[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kb + 64 * u + kq;
      if (VEC) {   // K % 4 == 0 and 16-byte aligned rows: the 4 columns are all in or all out
        in[u] = k < K;
        const int kc = min(k, K - 4);
        a[u] = *reinterpret_cast<const f32x4*>(pa + kc);
        b[u] = *reinterpret_cast<const f32x4*>(pb + kc);
      } else {
        in[u] = true;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int kc = min(k + q, K - 1);
          const float x = pa[kc], y = pb[kc];
          a[u][q] = k + q < K ? x : 0.f;
          b[u][q] = k + q < K ? y : 0.f;
        }
      }
    }
    // keep the loads of the batch ahead of its MFMAs
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool use_a = va && in[u], use_b = vb && in[u];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(use_a ? a[u][q] : 0.f, use_b ? b[u][q] : 0.f, acc, 0, 0, 0);
    }
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) red[wave][(4 * (lane >> 4) + v) * 16 + i] = acc[v];
  __syncthreads();
  const int r = threadIdx.x >> 4, c = threadIdx.x & 15;
  if (m0 + r < N1 && n0 + c < N2) {
    const float v = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
    g.out[z][(long long)(m0 + r) * N2 + n0 + c] = v + g.beta[z];
  }
}

template <bool VEC>
__global__ void __launch_bounds__(256) k_gram_small(GramBatch g, int N1, int N2, int tiles_n) {
  __shared__ float red[4][256];
  gram_small_block<VEC>(g, N1, N2, tiles_n, blockIdx.x, blockIdx.y, red);
}

hipError_t launch_gram(hipStream_t s, const GramBatch& g, int N1, int N2, int num_cu) {
  if (g.count <= 0) return hipSuccess;
  bool v = true;
  for (int z = 0; z < g.count; ++z)
    v = v && vec_ok(g.h1[z], g.K[z], g.K[z]) && vec_ok(g.h2[z], g.K[z], g.K[z]);
  if ((long long)cdiv(N1, CfgSmall::BM) * cdiv(N2, CfgSmall::BN) * g.count < num_cu) {
    const int tn = cdiv(N2, 16);
    const dim3 grid(cdiv(N1, 16) * tn, g.count);
    if (v)
      k_gram_small<true><<<grid, dim3(256), 0, s>>>(g, N1, N2, tn);
    else
      k_gram_small<false><<<grid, dim3(256), 0, s>>>(g, N1, N2, tn);
    return hipGetLastError();
  }
  bool dma = v;
  for (int z = 0; z < g.count; ++z)
    dma = dma && g.K[z] % 32 == 0 && dma_span_ok(g.K[z], g.K[z], 256);
  if (dma) return gram_vec<true, true>(s, g, N1, N2);
  return v ? gram_vec<true, false>(s, g, N1, N2) : gram_vec<false, false>(s, g, N1, N2);
}

// A backward layer of few tiles and the small-batch Grams in one launch: the first nbwd
// workgroups take the layer's tiles (which leave compute units idle), the others the 16 x 16
// Gram blocks (gblocks per layer input).
template <class Cfg, bool GVEC>
__global__ void __launch_bounds__(Cfg::THREADS)
k_dense_bwd_ko_gram(const float* __restrict__ G, const float* __restrict__ W, int R, int N, int K, EpiBwd epi,
                    int tiles_n, int nbwd, GramBatch g, int N1, int N2, int gtiles_n, int gblocks) {
  extern __shared__ float smem[];
  static_assert(Cfg::THREADS == 256, "the Gram blocks run on 256 threads");
  if ((int)blockIdx.x < nbwd) {
    dense_bwd_ko_tile<Cfg>(G, W, R, N, K, epi, tiles_n, blockIdx.x, smem);
  } else {
    const int b = blockIdx.x - nbwd;
    gram_small_block<GVEC>(g, N1, N2, gtiles_n, b % gblocks, b / gblocks, reinterpret_cast<float (*)[256]>(smem));
  }
}

static bool gram_small_fits(const GramBatch& g, int N1, int N2, int num_cu) {
  return g.count > 0 && (long long)cdiv(N1, 64) * cdiv(N2, 64) * g.count < num_cu;
}

static bool gram_batch_vec(const GramBatch& g) {
  bool v = true;
  for (int z = 0; z < g.count; ++z) v = v && vec_ok(g.h1[z], g.K[z], g.K[z]) && vec_ok(g.h2[z], g.K[z], g.K[z]);
  return v;
}

hipError_t launch_dense_bwd_w_gram(hipStream_t s, const float* G, const float* W, const float* dphi, int R, int N,
                                   int K, int O, float* out, const GramBatch& g, int N1, int N2, int num_cu) {
  if (O <= 0 || !dense_bwd_w_ok(G, W, R, N, K)) return hipErrorInvalidValue;
  const long long big_tiles = (long long)cdiv(R, 128) * cdiv(N, 128);
  if (big_tiles >= 512 || !gram_small_fits(g, N1, N2, num_cu)) {
    hipError_t e = launch_dense_bwd_w(s, G, W, dphi, R, N, K, O, out);
    return e != hipSuccess ? e : launch_gram(s, g, N1, N2, num_cu);
  }
  using Cfg = CfgSmall;
  EpiBwd epi{dphi, out, R, N, FastDiv((uint32_t)O)};
  const int tn = cdiv(N, Cfg::BN), tm = cdiv(R, Cfg::BM);
  const int gtn = cdiv(N2, 16), gblocks = cdiv(N1, 16) * gtn;
  const long long blocks = (long long)tm * tn + (long long)gblocks * g.count;
  constexpr int bytes = gemm_dma_smem_bytes<Cfg, 2>();
  static_assert(bytes >= 4 * 256 * 4, "the Gram blocks' partials fit the LDS of the tiles");
  auto go = [&](auto kern) -> hipError_t {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    kern<<<dim3((unsigned)blocks), dim3(Cfg::THREADS), bytes, s>>>(G, W, R, N, K, epi, tn, tm * tn, g, N1, N2, gtn,
                                                                    gblocks);
    return hipGetLastError();
  };
  return gram_batch_vec(g) ? go(k_dense_bwd_ko_gram<Cfg, true>) : go(k_dense_bwd_ko_gram<Cfg, false>);
}


// ------------------------------------------------------------------------------ fused contraction
// Stage the block of a Gram matrix that a tile touches (rows r cover samples r / O) into
// LDS: sg[a * S2 + b] = gram[n1lo + a][n2lo + b].  Ends with a barrier.
template <class Cfg>
__device__ __forceinline__ void stage_gram(const float* __restrict__ gram, int N2, int R1, int R2,
                                           FastDiv fO, int m0, int n0, float* sg, int& n1lo,
                                           int& n2lo, int& S2) {
  n1lo = (int)fO.div(m0);
  n2lo = (int)fO.div(n0);
  const int n1hi = (int)fO.div(min(m0 + Cfg::BM, R1) - 1);
  const int n2hi = (int)fO.div(min(n0 + Cfg::BN, R2) - 1);
  const int S1 = n1hi - n1lo + 1;
  S2 = n2hi - n2lo + 1;
  for (int q = threadIdx.x; q < S1 * S2; q += Cfg::THREADS) {
    const int a = q / S2, b = q - a * S2;
    sg[q] = gram[(long long)(n1lo + a) * N2 + n2lo + b];
  }
  __syncthreads();
}

// tot += gram_l[n1, n2] * (G1_l G2_l^T) over the tile at (m0, n0) (the scalar x1.x2 of Eq.
// mixed_product_example weights the cotangent product); the tile's Gram block is staged in the
// LDS tile area, free after the main loop.  Ends with a barrier.
template <class Cfg, bool VEC, bool DMA = false>
__device__ __forceinline__ void fcn_layer_term(const FcnContraction& c, int l, int N2, int R1, int R2, FastDiv fO,
                                               int m0, int n0, float* smem, f32x16 (&tot)[Cfg::FM][Cfg::FN]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM, wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
  const int K = c.K[l];
  LoadKInnerT<VEC> la{c.G1[l], R1, K, K};
  LoadKInnerT<VEC> lb{c.G2[l], R2, K, K};
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  if (DMA)
    gemm_mainloop_dma<Cfg, kSplitStages>(c.G1[l], K, R1, c.G2[l], K, R2, m0, n0, 0, K, smem, acc);
  else
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, K, smem, acc);
  int n1lo, n2lo, S2;
  stage_gram<Cfg>(c.gram[l], N2, R1, R2, fO, m0, n0, smem, n1lo, n2lo, S2);
#pragma unroll
  for (int fn = 0; fn < Cfg::FN; ++fn) {
    const int s = min(n0 + wn0 + fn * 32 + (lane & 31), R2 - 1);
    const int b = (int)fO.div(s) - n2lo;
#pragma unroll
    for (int fm = 0; fm < Cfg::FM; ++fm) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = min(m0 + wm0 + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3), R1 - 1);
        const int a = (int)fO.div(r) - n1lo;
        tot[fm][fn][v] += smem[a * S2 + b] * acc[fm][fn][v];
      }
      // keep one fragment's Gram values live at a time (register pressure)
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();
}

template <class Cfg, bool VEC>
__global__ void __launch_bounds__(Cfg::THREADS)
k_ntk_fcn(FcnContraction c, int N1, int N2, FastDiv fO, int symmetric, float* __restrict__ theta,
          int tiles_m, int tiles_n) {
  extern __shared__ float smem[];
  int tm, tn;
  if (symmetric) {
    tri_index(blockIdx.x, tiles_n, tm, tn);
  } else {
    tm = blockIdx.x / tiles_n;
    tn = blockIdx.x % tiles_n;
  }
  const int O = (int)fO.d;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int R1 = N1 * O, R2 = N2 * O;
  f32x16 tot[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(tot);
  for (int l = 0; l < c.L; ++l) fcn_layer_term<Cfg, VEC>(c, l, N2, R1, R2, fO, m0, n0, smem, tot);
  int n1lo, n2lo, S2;
  stage_gram<Cfg>(c.gram_readout, N2, R1, R2, fO, m0, n0, smem, n1lo, n2lo, S2);
  const bool mirror = symmetric && tm != tn;
  for_each_acc<Cfg>(tot, m0, n0, [&](int r, int s, float v) {
    if (r < R1 && s < R2) {
      const int n1 = (int)fO.div(r), o1 = r - n1 * O;
      const int n2 = (int)fO.div(s), o2 = s - n2 * O;
      if (o1 == o2) v += c.readout_scale * smem[(n1 - n1lo) * S2 + (n2 - n2lo)];
      theta[(((long long)n1 * N2 + n2) * O + o1) * O + o2] = v;
      if (mirror) theta[(((long long)n2 * N1 + n1) * O + o2) * O + o1] = v;
    }
  });
}

// ------------------------------------------------------------------------------ layer-split contraction
// Few output tiles (small batches): the layers are cut into NG contiguous groups, group g holding
// layers [g L / NG, (g + 1) L / NG), and workgroup (g, t) sums group g's terms of tile t, so the
// launch has T NG workgroups instead of T.  Each stores its partial tile (row-major 64 x 64) at
// part[(g T + t) 4096]; k_ntk_fcn_lreduce then adds the NG partials of a tile in group order and
// the readout summand and writes theta, so the result does not depend on the order in which the
// workgroups ran.
__device__ __forceinline__ void fcn_tile_coords(int t, int symmetric, int tiles_n, int& tm, int& tn) {
  if (symmetric) {
    tri_index(t, tiles_n, tm, tn);
  } else {
    tm = t / tiles_n;
    tn = t - tm * tiles_n;
  }
}

// The work of one tile (256 threads): the NG partial tiles added in group order, the readout
// summand, theta written from the LDS copy of the tile.  sg holds 64 x 64 floats, tile 64 x 65.
__device__ __forceinline__ void fcn_tile_reduce(const float* __restrict__ gram_readout, float readout_scale, int N1,
                                                int N2, FastDiv fO, int symmetric, int tiles_n, int T, int NG,
                                                const float* __restrict__ part, float* __restrict__ theta, int t,
                                                float* sg, float (*tile)[65]) {
  int tm, tn;
  fcn_tile_coords(t, symmetric, tiles_n, tm, tn);
  const int O = (int)fO.d;
  const int m0 = tm * 64, n0 = tn * 64;
  const int R1 = N1 * O, R2 = N2 * O;
  // the readout Gram block of the tile (rows r cover samples r / O)
  const int n1lo = (int)fO.div(m0), n2lo = (int)fO.div(n0);
  const int S1 = (int)fO.div(min(m0 + 64, R1) - 1) - n1lo + 1;
  const int S2 = (int)fO.div(min(n0 + 64, R2) - 1) - n2lo + 1;
  for (int q = threadIdx.x; q < S1 * S2; q += 256) {
    const int a = q / S2, b = q - a * S2;
    sg[q] = gram_readout[(long long)(n1lo + a) * N2 + n2lo + b];
  }
  // partial sums in group order: element e = 4 (threadIdx.x + 256 j) + i, j = 0..3, i = 0..3
  const float4* P = reinterpret_cast<const float4*>(part + (long long)t * 4096);
  const long long gstride = (long long)T * 1024;   // float4s between the partials of two groups
  float4 v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = P[threadIdx.x + 256 * j];
  // the groups four at a time, all their loads in flight together (a group past NG reads the
  // last one again and is not added)
  for (int g0 = 1; g0 < NG; g0 += 4) {
    float4 w[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const long long g = min(g0 + u, NG - 1);
#pragma unroll
      for (int j = 0; j < 4; ++j) w[u][j] = P[g * gstride + threadIdx.x + 256 * j];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (g0 + u < NG) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[j].x += w[u][j].x;
          v[j].y += w[u][j].y;
          v[j].z += w[u][j].z;
          v[j].w += w[u][j].w;
        }
      }
  }
  __syncthreads();   // sg complete
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * (threadIdx.x + 256 * j);
    const int rl = e >> 6, sl = e & 63;
    const float vv[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
    const int r = m0 + rl;
    const int n1 = (int)fO.div(min(r, R1 - 1)), o1 = r - n1 * O;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int s = n0 + sl + i;
      const int n2 = (int)fO.div(min(s, R2 - 1)), o2 = s - n2 * O;
      float x = vv[i];
      if (o1 == o2 && r < R1 && s < R2) x += readout_scale * sg[(n1 - n1lo) * S2 + (n2 - n2lo)];
      tile[rl][sl + i] = x;
    }
  }
  __syncthreads();
  // direct block: consecutive threads take consecutive columns s = (n2, o2)
  for (int e = threadIdx.x; e < 4096; e += 256) {
    const int rl = e >> 6, sl = e & 63;
    const int r = m0 + rl, s = n0 + sl;
    if (r < R1 && s < R2) {
      const int n1 = (int)fO.div(r), o1 = r - n1 * O;
      const int n2 = (int)fO.div(s), o2 = s - n2 * O;
      theta[(((long long)n1 * N2 + n2) * O + o1) * O + o2] = tile[rl][sl];
    }
  }
  if (!(symmetric && tm != tn)) return;
  // mirrored block theta[n2][n1][o2][o1]: consecutive threads take consecutive rows r = (n1, o1)
  for (int e = threadIdx.x; e < 4096; e += 256) {
    const int sl = e >> 6, rl = e & 63;
    const int r = m0 + rl, s = n0 + sl;
    if (r < R1 && s < R2) {
      const int n1 = (int)fO.div(r), o1 = r - n1 * O;
      const int n2 = (int)fO.div(s), o2 = s - n2 * O;
      theta[(((long long)n2 * N1 + n1) * O + o2) * O + o1] = tile[rl][sl];
    }
  }
}

template <class Cfg, bool VEC, bool DMA>
__global__ void __launch_bounds__(Cfg::THREADS)
k_ntk_fcn_lpart(FcnContraction c, int N1, int N2, FastDiv fO, int symmetric, int tiles_n, int T, int NG,
                float* __restrict__ part) {
  extern __shared__ float smem[];
  // the (group, tile) list in group-major order, in contiguous ranges per XCD: an XCD's
  // workgroups read the cotangents of one or two layer groups through its L2
  int blk;
  if (!xcd_block(blockIdx.x, T * NG, blk)) return;
  const int g = blk / T, t = blk - g * T;
  int tm, tn;
  fcn_tile_coords(t, symmetric, tiles_n, tm, tn);
  const int O = (int)fO.d;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int R1 = N1 * O, R2 = N2 * O;
  const int l0 = (int)((long long)g * c.L / NG), l1 = (int)((long long)(g + 1) * c.L / NG);
  f32x16 tot[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(tot);
  for (int l = l0; l < l1; ++l) fcn_layer_term<Cfg, VEC, DMA>(c, l, N2, R1, R2, fO, m0, n0, smem, tot);
  float* P = part + ((long long)g * T + t) * (Cfg::BM * Cfg::BN);
  for_each_acc<Cfg>(tot, 0, 0, [&](int r, int s, float v) { P[r * Cfg::BN + s] = v; });
}

// One workgroup per tile.  Each thread adds 16 elements (four float4s) of the tile's NG partials
// in group order, the four loads of one partial in flight together, adds the readout summand and
// stages the result in LDS; theta is then written in runs of O consecutive floats: the direct
// block in row order, the mirrored one (symmetric schedule) in column order.
__global__ void __launch_bounds__(256)
k_ntk_fcn_lreduce(const float* __restrict__ gram_readout, float readout_scale, int N1, int N2, FastDiv fO,
                  int symmetric, int tiles_n, int T, int NG, const float* __restrict__ part,
                  float* __restrict__ theta) {
  __shared__ float sg[64 * 64];
  __shared__ float tile[64][65];
  fcn_tile_reduce(gram_readout, readout_scale, N1, N2, fO, symmetric, tiles_n, T, NG, part, theta, blockIdx.x, sg,
                  tile);
}

// ------------------------------------------------------------------------------ stream-K contraction
// The contraction's work is T tiles x L layers over P persistent workgroups (kSkPerCu per
// compute unit; P = 8 * P8, P8 per XCD).  Workgroup ids are dispatched round robin over the 8 XCDs,
// each with its own L2, so the schedule is built per XCD:
//   * tile order: the tile grid is cut into 8 bands of columns and ordered band by band,
//     row by row inside a band; XCD x takes the x-th contiguous eighth of that order, so its
//     workgroups share the B panels of a few columns for the whole launch;
//   * data-parallel rounds: the XCD's P8 workgroups take whole tiles, P8 per round (the
//     tiles of one round are neighbours and progress through the layers together);
//   * stream-K tail: the XCD's last (T_x mod P8) tiles are cut into (tile, layer) units and
//     split into P8 equal contiguous ranges.  A range covering all layers of a tile writes
//     theta; a split tile's partial sums go to `part` (slot 0: the first tile of a range,
//     slot 1: its last) and k_ntk_fcn_fixup adds them in range order.
// No workgroup waits for another; the summation order is fixed for a given device.
// Final epilogue of a tile: add the readout summand, write theta (and its mirror).
template <class Cfg>
__device__ __forceinline__ void fcn_tile_out(f32x16 (&tot)[Cfg::FM][Cfg::FN], const float* gram_readout,
                                             float rscale, int N1, int N2, FastDiv fO, int R1, int R2,
                                             int m0, int n0, bool mirror, float* smem,
                                             float* __restrict__ theta) {
  const int O = (int)fO.d;
  int n1lo, n2lo, S2;
  stage_gram<Cfg>(gram_readout, N2, R1, R2, fO, m0, n0, smem, n1lo, n2lo, S2);
  for_each_acc<Cfg>(tot, m0, n0, [&](int r, int s, float v) {
    if (r < R1 && s < R2) {
      const int n1 = (int)fO.div(r), o1 = r - n1 * O;
      const int n2 = (int)fO.div(s), o2 = s - n2 * O;
      if (o1 == o2) v += rscale * smem[(n1 - n1lo) * S2 + (n2 - n2lo)];
      theta[(((long long)n1 * N2 + n2) * O + o1) * O + o2] = v;
      if (mirror) theta[(((long long)n2 * N1 + n1) * O + o2) * O + o1] = v;
    }
  });
  __syncthreads();
}

// tot += sum over layers [l0, l1) of gram_l (.) (G1_l G2_l^T) for the tile at (m0, n0).
// DMA: direct-to-LDS main loop (every K % 32 == 0, VEC operands).
template <class Cfg, bool VEC, bool DMA>
__device__ __forceinline__ void fcn_tile_layers(const FcnContraction& c, int l0, int l1, int N2,
                                                FastDiv fO, int R1, int R2, int m0, int n0,
                                                float* smem, f32x16 (&tot)[Cfg::FM][Cfg::FN]) {
  const int lane_id = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM, wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
  for (int l = l0; l < l1; ++l) {
    const int K = c.K[l];
    f32x16 acc[Cfg::FM][Cfg::FN];
    zero_acc<Cfg>(acc);
    if (DMA) {
      gemm_mainloop_dma<Cfg, kSkStages>(c.G1[l], K, R1, c.G2[l], K, R2, m0, n0, 0, K, smem, acc);
    } else {
      LoadKInnerT<VEC> la{c.G1[l], R1, K, K};
      LoadKInnerT<VEC> lb{c.G2[l], R2, K, K};
      gemm_mainloop<Cfg>(la, lb, m0, n0, 0, K, smem, acc);
    }
    int n1lo, n2lo, S2;
    stage_gram<Cfg>(c.gram[l], N2, R1, R2, fO, m0, n0, smem, n1lo, n2lo, S2);
    // The Gram addresses below do not change from layer to layer; computed once they would
    // hold ~30 registers through the main loop.  An opaque copy of the lane index keeps
    // them inside the epilogue.
    int lane = lane_id;
    asm volatile("" : "+v"(lane));
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn) {
      const int sc = min(n0 + wn0 + fn * 32 + (lane & 31), R2 - 1);
      const int b = (int)fO.div(sc) - n2lo;
#pragma unroll
      for (int fm = 0; fm < Cfg::FM; ++fm) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = min(m0 + wm0 + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3), R1 - 1);
          const int a = (int)fO.div(r) - n1lo;
          tot[fm][fn][v] += smem[a * S2 + b] * acc[fm][fn][v];
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();
  }
}

// kSkPerCu workgroups per compute unit must be resident together: the register budget is that
// of kSkPerCu * THREADS / 256 waves per SIMD
template <class Cfg, bool VEC, bool DMA>
__global__ void __launch_bounds__(Cfg::THREADS, kSkPerCu * Cfg::THREADS / 256)
k_ntk_fcn_sk(FcnContraction c, int N1, int N2, FastDiv fO, int symmetric, float* __restrict__ theta,
             int tiles_m, int tiles_n, int T, int P, float* __restrict__ part) {
  extern __shared__ float smem[];
  const int bid = blockIdx.x;
  const int P8 = P >> 3;
  const int x = bid & 7, j = bid >> 3;        // XCD and workgroup index inside it
  const int lam = x * P8 + j;                 // partial-buffer owner id
  const int L = c.L;
  const SkShare sh = sk_share(x, T, P8, L);
  const int O = (int)fO.d;
  const int R1 = N1 * O, R2 = N2 * O;
  // The XCD's data-parallel rounds (whole tiles), then its stream-K range of (tile, layer)
  // units, as one loop so that the main loop is instantiated once.
  const long long beg = sk_start(j, sh.U, P8), end = sk_start(j + 1, sh.U, P8);
  int i = 0;
  long long u = beg;
  while (true) {
    int t, ts = 0, l0 = 0, l1 = L;
    if (i < sh.rounds) {
      t = sh.base + i * P8 + j;
    } else {
      if (u >= end) break;
      ts = (int)(u / L);
      l0 = (int)(u - (long long)ts * L);
      l1 = (int)min((long long)L, l0 + (end - u));
      t = sh.first_sk + ts;
    }
    int tm, tn;
    tile_coords(t, symmetric, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
    f32x16 tot[Cfg::FM][Cfg::FN];
    zero_acc<Cfg>(tot);
    fcn_tile_layers<Cfg, VEC, DMA>(c, l0, l1, N2, fO, R1, R2, m0, n0, smem, tot);
    if (l0 == 0 && l1 == L) {
      fcn_tile_out<Cfg>(tot, c.gram_readout, c.readout_scale, N1, N2, fO, R1, R2, m0, n0, symmetric && tm != tn, smem,
                        theta);
    } else {
      float* dst = part + ((long long)lam * 2 + sk_slot(beg, L, ts)) * (Cfg::BM * Cfg::BN);
      int z = 0;   // opaque zero: keeps the 32 store offsets from being computed up front
      asm volatile("" : "+v"(z));
      for_each_acc<Cfg>(tot, z, z, [&](int ii, int jj, float v) { dst[ii * Cfg::BN + jj] = v; });
    }
    if (i < sh.rounds) ++i;
    else u += l1 - l0;
  }
}

// Fixup of the stream-K tails.  Boundary j = 1..P8-1 of XCD x owns a tile when it falls inside
// it and is the first boundary inside it (sk_fixup_tile); kFixupSplit workgroups share that
// tile, each thread adds the partial sums of one float4 of it (ranges in order), adds the
// readout summand and writes theta.
constexpr int kFixupSplit = 16;
template <class Cfg>
__global__ void __launch_bounds__(256)
k_ntk_fcn_fixup(int L, const float* __restrict__ gram_readout, float rscale, int N1, int N2, FastDiv fO,
                int symmetric, float* __restrict__ theta, int tiles_m, int tiles_n, int T, int P,
                const float* __restrict__ part) {
  static_assert(Cfg::BM * Cfg::BN == kFixupSplit * 256 * 4, "one float4 per thread");
  const int P8 = P >> 3;
  const int blk = blockIdx.x / kFixupSplit, sub = blockIdx.x % kFixupSplit;
  const int x = blk / (P8 - 1), j = blk % (P8 - 1) + 1;
  const SkShare sh = sk_share(x, T, P8, L);
  const int ts = sk_fixup_tile(sh, j, P8, L);
  if (ts < 0) return;
  int tm, tn;
  tile_coords(sh.first_sk + ts, symmetric, tiles_m, tiles_n, tm, tn);
  const int e0 = (sub * 256 + threadIdx.x) * 4;
  const long long tile_end = (long long)(ts + 1) * L;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  long long qb = sk_start(j - 1, sh.U, P8);
  for (int q = j - 1; q < P8 && qb < tile_end; ++q) {
    const long long qe = sk_start(q + 1, sh.U, P8);
    if (qe > qb) {   // an empty range wrote nothing
      const float4 p = *reinterpret_cast<const float4*>(
          part + ((long long)(x * P8 + q) * 2 + sk_slot(qb, L, ts)) * (Cfg::BM * Cfg::BN) + e0);
      v.x += p.x;
      v.y += p.y;
      v.z += p.z;
      v.w += p.w;
    }
    qb = qe;
  }
  const int O = (int)fO.d;
  const int R1 = N1 * O, R2 = N2 * O;
  const bool mirror = symmetric && tm != tn;
  const int i = e0 / Cfg::BN, jj = e0 - i * Cfg::BN;
  const int r = tm * Cfg::BM + i;
  if (r >= R1) return;
  const int n1 = (int)fO.div(r), o1 = r - n1 * O;
  const float vals[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int s = tn * Cfg::BN + jj + k;
    if (s < R2) {
      const int n2 = (int)fO.div(s), o2 = s - n2 * O;
      float w = vals[k];
      if (o1 == o2) w += rscale * gram_readout[(long long)n1 * N2 + n2];
      theta[(((long long)n1 * N2 + n2) * O + o1) * O + o2] = w;
      if (mirror) theta[(((long long)n2 * N1 + n1) * O + o2) * O + o1] = w;
    }
  }
}

// The staged Gram block is at most (BM/O + 2) x (BN/O + 2) floats, and BM x BN for O = 1;
// it must fit the LDS tile area.
template <class Cfg, class L>
constexpr bool gram_block_fits() {
  return (Cfg::BM + 1) * (Cfg::BN + 1) <= gemm_smem_bytes<Cfg, L, L>() / 4;
}

long long ntk_fcn_part_floats(int num_cu) {
  return (long long)kSkPerCu * num_cu * 2 * CfgSK::BM * CfgSK::BN;
}

static bool fcn_uses_stream_k(int L, long long big_tiles, int num_cu, bool part) {
  // stream-K when there are at least as many whole tiles as persistent workgroups (P must be
  // a multiple of 8 for the XCD-aware range order)
  return L >= 1 && part && num_cu >= 16 && num_cu % 8 == 0 && big_tiles >= kSkPerCu * num_cu;
}

// Few output tiles: the number of layer groups of the layer-split contraction (>= 2), or 0 when
// that form does not apply.
static int fcn_split_groups(long long R1, long long R2, int L, int symmetric, int num_cu, bool part) {
  const long long big_tiles = (long long)cdiv(R1, 128) * cdiv(R2, 128);
  if (!part || L < 2 || fcn_uses_stream_k(L, big_tiles, num_cu, part) || big_tiles >= 512) return 0;
  // fewer 64 x 64 tiles than two per compute unit: about four workgroups per compute unit in
  // all, as far as the partial tiles fit the buffer
  const long long ts_m = cdiv(R1, 64), ts_n = cdiv(R2, 64);
  const long long Ts = symmetric ? ts_n * (ts_n + 1) / 2 : ts_m * ts_n;
  if (Ts >= 2LL * num_cu) return 0;
  long long NG = std::min<long long>(L, (4LL * num_cu + Ts - 1) / Ts);
  NG = std::min<long long>(NG, ntk_fcn_part_floats(num_cu) / (Ts * 4096));
  return NG >= 2 ? (int)NG : 0;
}

hipError_t launch_ntk_fcn(hipStream_t s, const FcnContraction& c, int N1, int N2, int O,
                          int symmetric, float* theta, int num_cu, float* part) {
  int R1, R2;
  if (!to_int((long long)N1 * O, R1) || !to_int((long long)N2 * O, R2)) return hipErrorInvalidValue;
  bool v = true;
  for (int l = 0; l < c.L; ++l)
    v = v && vec_ok(c.G1[l], c.K[l], c.K[l]) && vec_ok(c.G2[l], c.K[l], c.K[l]);
  auto go = [&](auto cfg_tag, auto vec_tag) -> hipError_t {
    using Cfg = decltype(cfg_tag);
    constexpr bool VEC = decltype(vec_tag)::value;
    using L = LoadKInnerT<VEC>;
    static_assert(gram_block_fits<Cfg, L>(), "Gram block must fit the LDS tile area");
    const int tm = cdiv(R1, Cfg::BM), tn = cdiv(R2, Cfg::BN);
    const int tiles = symmetric ? tn * (tn + 1) / 2 : tm * tn;
    hipError_t e = set_smem<Cfg, L, L>((const void*)k_ntk_fcn<Cfg, VEC>);
    if (e != hipSuccess) return e;
    k_ntk_fcn<Cfg, VEC><<<dim3(tiles), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, L, L>(), s>>>(
        c, N1, N2, FastDiv((uint32_t)O), symmetric, theta, tm, tn);
    return hipGetLastError();
  };
  bool dma = v;
  for (int l = 0; l < c.L; ++l) dma = dma && c.K[l] % 32 == 0 && dma_span_ok(c.K[l], c.K[l], 256);
  auto go_sk = [&](auto vec_tag, auto dma_tag) -> hipError_t {
    using Cfg = CfgSK;
    constexpr bool VEC = decltype(vec_tag)::value;
    constexpr bool DMA = decltype(dma_tag)::value;
    using L = LoadKInnerT<VEC>;
    const int tm = cdiv(R1, Cfg::BM), tn = cdiv(R2, Cfg::BN);
    const int T = symmetric ? tn * (tn + 1) / 2 : tm * tn;
    const int P = kSkPerCu * num_cu;
    // LDS: the main loop's stages, or the Gram block of a tile if larger
    constexpr int loop_bytes = DMA ? gemm_dma_smem_bytes<Cfg, kSkStages>() : gemm_smem_bytes<Cfg, L, L>();
    constexpr int gram_bytes = (Cfg::BM + 1) * (Cfg::BN + 1) * 4;
    constexpr int bytes = loop_bytes > gram_bytes ? loop_bytes : gram_bytes;
    static_assert(kSkPerCu * bytes <= 160 * 1024, "the workgroups of one CU must fit its LDS");
    hipError_t e = hipFuncSetAttribute((const void*)k_ntk_fcn_sk<Cfg, VEC, DMA>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    const FastDiv fO((uint32_t)O);
    k_ntk_fcn_sk<Cfg, VEC, DMA><<<dim3(P), dim3(Cfg::THREADS), bytes, s>>>(
        c, N1, N2, fO, symmetric, theta, tm, tn, T, P, part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_ntk_fcn_fixup<Cfg><<<dim3(8 * (P / 8 - 1) * kFixupSplit), dim3(256), 0, s>>>(
        c.L, c.gram_readout, c.readout_scale, N1, N2, fO, symmetric, theta, tm, tn, T, P, part);
    return hipGetLastError();
  };
  const long long big_tiles = (long long)cdiv(R1, 128) * cdiv(R2, 128);
  if (fcn_uses_stream_k(c.L, big_tiles, num_cu, part != nullptr))
    return dma ? go_sk(TrueT{}, TrueT{}) : (v ? go_sk(TrueT{}, FalseT{}) : go_sk(FalseT{}, FalseT{}));
  if (big_tiles >= 512) return v ? go(CfgBig8{}, TrueT{}) : go(CfgBig8{}, FalseT{});
  const int NG = fcn_split_groups(R1, R2, c.L, symmetric, num_cu, part != nullptr);
  auto go_split = [&](auto vec_tag, auto dma_tag) -> hipError_t {
    using Cfg = CfgSmall;
    constexpr bool VEC = decltype(vec_tag)::value;
    constexpr bool DMA = decltype(dma_tag)::value;
    using L = LoadKInnerT<VEC>;
    constexpr int bytes = DMA ? gemm_dma_smem_bytes<Cfg, kSplitStages>() : gemm_smem_bytes<Cfg, L, L>();
    static_assert(64 * 64 <= bytes / 4, "Gram block must fit the LDS tile area");
    const int tm = cdiv(R1, 64), tn = cdiv(R2, 64);
    const int T = symmetric ? tn * (tn + 1) / 2 : tm * tn;
    const FastDiv fO((uint32_t)O);
    hipError_t e = hipFuncSetAttribute((const void*)k_ntk_fcn_lpart<Cfg, VEC, DMA>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    k_ntk_fcn_lpart<Cfg, VEC, DMA><<<dim3(8 * cdiv((long long)T * NG, 8)), dim3(Cfg::THREADS), bytes, s>>>(
        c, N1, N2, fO, symmetric, tn, T, NG, part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_ntk_fcn_lreduce<<<dim3(T), dim3(256), 0, s>>>(c.gram_readout, c.readout_scale, N1, N2, fO, symmetric, tn, T,
                                                    NG, part, theta);
    return hipGetLastError();
  };
  if (NG >= 2) return dma ? go_split(TrueT{}, TrueT{}) : (v ? go_split(TrueT{}, FalseT{}) : go_split(FalseT{}, FalseT{}));
  return v ? go(CfgSmall{}, TrueT{}) : go(CfgSmall{}, FalseT{});
}

}  // namespace ntk
