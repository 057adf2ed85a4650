// kernels_diag.hip -- the output-axis and batch-axis variants of Theta.
//
// Section 3 of the paper defines Theta over all pairs of inputs and all pairs of outputs; the
// variants below keep a part of it (appendix "Pseudo-NTK" and the batch diagonal Theta(x, x)):
//   * trace over the outputs:     sum_o Theta(x1, x2)[o, o]       [N1, N2]
//   * one logit o*:               Theta(x1, x2)[o*, o*]            [N1, N2]
//   * batch diagonal:             Theta(x1_n, x2_n)                [N, O, O] (or [N] traced)
// The first two are the full contraction with one output (the trace contracts the cotangent
// rows of all O outputs as one row of O*K columns), run by the contraction kernels with O = 1.
// The batch diagonal needs, per sample, the layer-input scalars d_l[n] = h1_l[n] . h2_l[n]
// (+1 with a bias) and the per-sample cotangent products; the kernels here compute them.
#include "gemm_core.hpp"
#include "launch.hpp"

namespace ntk {

// ------------------------------------------------------------------------------ block reduction
// Sum of one float per thread over a 256-thread block, in a fixed order.  Every thread gets it.
__device__ __forceinline__ float block_sum_256(float v, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();                 // `red` may still be read by a previous call
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// a[0..K) . b[0..K) by one 256-thread block; float4 loads when both rows are 16-byte aligned.
__device__ __forceinline__ float block_dot(const float* a, const float* b, long long K, float* red) {
  float acc = 0.f;
  if (((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b)) & 15) == 0) {
    const long long K4 = K >> 2;
    const float4* a4 = reinterpret_cast<const float4*>(a);
    const float4* b4 = reinterpret_cast<const float4*>(b);
    for (long long i = threadIdx.x; i < K4; i += 256) {
      const float4 x = a4[i], y = b4[i];
      acc += x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
    }
    for (long long i = (K4 << 2) + threadIdx.x; i < K; i += 256) acc += a[i] * b[i];
  } else {
    for (long long i = threadIdx.x; i < K; i += 256) acc += a[i] * b[i];
  }
  return block_sum_256(acc, red);
}

// ------------------------------------------------------------------------------ row dots
// out_j[n] = a_j[n] . b_j[n] + beta_j, one block per (n, j).
__global__ void __launch_bounds__(256) k_rowdot_batch(RowdotBatch r) {
  __shared__ float red[4];
  const int n = blockIdx.x, j = blockIdx.y;
  const long long K = r.K[j];
  const float v = block_dot(r.a[j] + n * K, r.b[j] + n * K, K, red);
  if (threadIdx.x == 0) r.out[j][n] = v + r.beta[j];
}

hipError_t launch_rowdot(hipStream_t s, const RowdotBatch& r, int N) {
  if (r.count <= 0 || N <= 0) return hipSuccess;
  k_rowdot_batch<<<dim3(N, r.count), dim3(256), 0, s>>>(r);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------ traced diagonal
// theta[n] (+)= sum_l w_l[n] (A_l[n] . B_l[n]) + readout_scale * readout[n], one block per n.
__global__ void __launch_bounds__(256) k_ntk_diag_flat(DiagTerms t, int accumulate, float* __restrict__ theta) {
  __shared__ float red[4];
  const int n = blockIdx.x;
  float tot = 0.f;
  for (int l = 0; l < t.count; ++l) {
    const long long K = t.K[l];
    const float d = block_dot(t.A[l] + n * K, t.B[l] + n * K, K, red);
    tot += (t.w[l] ? t.w[l][n] : 1.f) * d;
  }
  if (threadIdx.x == 0) {
    if (t.readout) tot += t.readout_scale * t.readout[n];
    theta[n] = accumulate ? theta[n] + tot : tot;
  }
}

// ------------------------------------------------------------------------------ O x O diagonal
// theta[n, o1, o2] (+)= sum_l w_l[n] (A_l[n] B_l[n]^T)[o1, o2] + readout_scale * readout[n] delta,
// with A_l[n] the O x K_l block at A_l + n O K_l.  One wave per (n, 32 x 32 tile of outputs).
using CfgDiag = TileCfg<32, 32, 32, 32, 32>;

template <bool VEC>
__global__ void __launch_bounds__(64)
k_ntk_diag_block(DiagTerms t, int O, int tiles_o, int accumulate, float* __restrict__ theta) {
  using Cfg = CfgDiag;
  extern __shared__ float smem[];
  const int tiles = tiles_o * tiles_o;
  const int n = blockIdx.x / tiles, tt = blockIdx.x % tiles;
  const int m0 = (tt / tiles_o) * Cfg::BM, n0 = (tt % tiles_o) * Cfg::BN;
  f32x16 tot[1][1];
  zero_acc<Cfg>(tot);
  for (int l = 0; l < t.count; ++l) {
    const long long K = t.K[l];
    LoadKInnerT<VEC> la{t.A[l] + (long long)n * O * K, O, (int)K, K};
    LoadKInnerT<VEC> lb{t.B[l] + (long long)n * O * K, O, (int)K, K};
    f32x16 acc[1][1];
    zero_acc<Cfg>(acc);
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, (int)K, smem, acc);
    const float w = t.w[l] ? t.w[l][n] : 1.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) tot[0][0][v] += w * acc[0][0][v];
    __syncthreads();
  }
  const float r = t.readout ? t.readout_scale * t.readout[n] : 0.f;
  float* out = theta + (long long)n * O * O;
  for_each_acc<Cfg>(tot, m0, n0, [&](int o1, int o2, float v) {
    if (o1 < O && o2 < O) {
      if (o1 == o2) v += r;
      float* dst = out + (long long)o1 * O + o2;
      *dst = accumulate ? *dst + v : v;
    }
  });
}

// K-segmented form: segment g covers columns [kb, ke) of one term l; every (segment, sample,
// tile) is one wave writing w_l[n] times its partial product to part[g][n][o1][o2], and
// k_ntk_diag_reduce adds the segments in order.
struct DiagSegs {
  int base[kMaxLayers + 1];   // first segment of term l; base[count] = number of segments
  int len[kMaxLayers];        // columns per segment of term l (a multiple of the K tile)
};

template <bool VEC>
__global__ void __launch_bounds__(64)
k_ntk_diag_seg(DiagTerms t, DiagSegs sg, int N, int O, int tiles_o, float* __restrict__ part) {
  using Cfg = CfgDiag;
  extern __shared__ float smem[];
  const int tiles = tiles_o * tiles_o;
  const int per_seg = N * tiles;
  const int g = blockIdx.x / per_seg, rem = blockIdx.x % per_seg;
  const int n = rem / tiles, tt = rem % tiles;
  int l = 0;
  while (sg.base[l + 1] <= g) ++l;
  const int K = (int)t.K[l];
  const int kb = (g - sg.base[l]) * sg.len[l], ke = min(K, kb + sg.len[l]);
  const int m0 = (tt / tiles_o) * Cfg::BM, n0 = (tt % tiles_o) * Cfg::BN;
  LoadKInnerT<VEC> la{t.A[l] + (long long)n * O * K, O, K, K};
  LoadKInnerT<VEC> lb{t.B[l] + (long long)n * O * K, O, K, K};
  f32x16 acc[1][1];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, kb, ke, smem, acc);
  const float w = t.w[l] ? t.w[l][n] : 1.f;
  float* out = part + ((long long)g * N + n) * O * O;
  for_each_acc<Cfg>(acc, m0, n0, [&](int o1, int o2, float v) {
    if (o1 < O && o2 < O) out[(long long)o1 * O + o2] = w * v;
  });
}

__global__ void __launch_bounds__(256)
k_ntk_diag_reduce(const float* __restrict__ part, int nseg, int N, int O, const float* __restrict__ readout,
                  float rscale, int accumulate, float* __restrict__ theta) {
  const long long total = (long long)N * O * O;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    int g = 0;
    for (; g + 4 <= nseg; g += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] += part[(long long)(g + u) * total + i];
    }
    for (; g < nseg; ++g) acc[0] += part[(long long)g * total + i];
    float v = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    const int n = (int)(i / ((long long)O * O));
    const int q = (int)(i - (long long)n * O * O);
    if (readout && q / O == q % O) v += rscale * readout[n];
    theta[i] = accumulate ? theta[i] + v : v;
  }
}

hipError_t launch_ntk_diag(hipStream_t s, const DiagTerms& t, int N, int O, int accumulate,
                           float* theta, float* part, long long part_capacity) {
  if (N <= 0) return hipSuccess;
  if (O == 0) {   // traced: one value per sample
    k_ntk_diag_flat<<<dim3(N), dim3(256), 0, s>>>(t, accumulate, theta);
    return hipGetLastError();
  }
  bool v = true;
  for (int l = 0; l < t.count; ++l) v = v && vec_ok(t.A[l], t.K[l], t.K[l]) && vec_ok(t.B[l], t.K[l], t.K[l]);
  const int tiles_o = (O + CfgDiag::BM - 1) / CfgDiag::BM;
  using L = LoadKInnerT<true>;
  constexpr int bytes = gemm_smem_bytes<CfgDiag, L, L>();
  // segments: about 2048 waves in all, at least 8 K tiles per segment, whole terms at least
  const long long waves_per_seg = (long long)N * tiles_o * tiles_o;
  long long Ktot = 0;
  for (int l = 0; l < t.count; ++l) Ktot += t.K[l];
  const long long want = std::max<long long>(1, (2048 + waves_per_seg - 1) / waves_per_seg);
  DiagSegs sg{};
  int nseg = 0;
  for (int l = 0; l < t.count; ++l) {
    const long long K = t.K[l];
    long long nl = std::max<long long>(1, (want * K + Ktot - 1) / std::max<long long>(Ktot, 1));
    nl = std::min<long long>(nl, std::max<long long>(1, K / (8 * CfgDiag::BK)));
    long long len = (K + nl - 1) / nl;
    len = ((len + CfgDiag::BK - 1) / CfgDiag::BK) * CfgDiag::BK;
    sg.base[l] = nseg;
    sg.len[l] = (int)len;
    nseg += (int)((K + len - 1) / len);
  }
  sg.base[t.count] = nseg;
  const bool seg_ok = part && t.count > 0 && (long long)nseg * N * O * O <= part_capacity &&
                      Ktot < (1LL << 31);
  if (!seg_ok) {
    if (v)
      k_ntk_diag_block<true><<<dim3(N * tiles_o * tiles_o), dim3(CfgDiag::THREADS), bytes, s>>>(
          t, O, tiles_o, accumulate, theta);
    else
      k_ntk_diag_block<false><<<dim3(N * tiles_o * tiles_o), dim3(CfgDiag::THREADS), bytes, s>>>(
          t, O, tiles_o, accumulate, theta);
    return hipGetLastError();
  }
  const long long grid = (long long)nseg * waves_per_seg;
  if (v)
    k_ntk_diag_seg<true><<<dim3((unsigned)grid), dim3(CfgDiag::THREADS), bytes, s>>>(t, sg, N, O, tiles_o, part);
  else
    k_ntk_diag_seg<false><<<dim3((unsigned)grid), dim3(CfgDiag::THREADS), bytes, s>>>(t, sg, N, O, tiles_o, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long long total = (long long)N * O * O;
  const int blocks = (int)std::min<long long>((total + 255) / 256, 4096);
  k_ntk_diag_reduce<<<dim3(blocks), dim3(256), 0, s>>>(part, nseg, N, O, t.readout, t.readout_scale,
                                                       accumulate, theta);
  return hipGetLastError();
}

}  // namespace ntk
