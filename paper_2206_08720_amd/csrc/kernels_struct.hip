// kernels_struct.hip -- the further structure rules of the paper's appendix on structured
// derivatives, for convolutional models:
//
//   * depthwise 3x3 convolution: dz/dw is block-diagonal over channels (channel c's filter
//     feeds only output channel c), so its weight-space cotangent is, per row (n, o) and
//     channel c, nine pixel sums  sum_p G[p, c] x[p + offset(t), c]  -- 9*C columns, not a
//     matrix product;
//   * per-channel scale z = x * w[c]: block-diagonal over channels and output block-tiled over
//     the pixels (the same w[c] multiplies every pixel): one pixel sum sum_p G[p, c] x[p, c];
//   * a bias broadcast over the pixels (convolution, depthwise or scale layer): output
//     block-tiled, its Jacobian rows are the cotangents summed over the pixels;
//   * 2x2 average pooling (stride 2): no parameters; it only moves the cotangents.
//
// These columns join the outside-in weight-space cotangents of the 3x3 convolutions in one
// matrix J per call, whose product J1 J2^T the split-K contraction forms.  Every kernel here is
// a memory-bound elementwise or stencil pass over NHWC planes: a lane owns V consecutive
// channels of one pixel (V = 4 when C % 4 == 0 and the buffers are 16-byte aligned, else 1), so a
// wave reads contiguous channel runs.  Forward pre-activations are accumulated in fp64 (the
// activation's decision is then that of the exact pre-activation of the fp32-stored inputs, as
// in the dense and convolution forward kernels); cotangents are fp32.
#include <algorithm>

#include "../../include/ntk.h"
#include "gemm_core.hpp"
#include "index_math.hpp"
#include "launch_struct.hpp"

namespace ntk {
namespace {

inline int cdiv_i(long long a, long long b) { return (int)((a + b - 1) / b); }
inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <int V>
struct Vf {
  float v[V];
};

template <int V>
__device__ __forceinline__ Vf<V> ldv(const float* __restrict__ p) {
  Vf<V> r;
  if constexpr (V == 4) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    r.v[0] = t.x;
    r.v[1] = t.y;
    r.v[2] = t.z;
    r.v[3] = t.w;
  } else {
    r.v[0] = *p;
  }
  return r;
}

template <int V>
__device__ __forceinline__ void stv(float* __restrict__ p, const Vf<V>& r) {
  if constexpr (V == 4)
    *reinterpret_cast<float4*>(p) = make_float4(r.v[0], r.v[1], r.v[2], r.v[3]);
  else
    *p = r.v[0];
}

// act and act' of a pre-activation accumulated in fp64: the ReLU decides on the fp64 value,
// erf is evaluated at its fp32 rounding
__device__ __forceinline__ void act_pair(int act, double z, float& h, float& d) {
  if (act == NTK_ACT_RELU) {
    h = z > 0.0 ? (float)z : 0.f;
    d = z > 0.0 ? 1.f : 0.f;
  } else {
    const float zf = (float)z;
    h = act_fwd(act, zf);
    d = act_deriv(act, zf);
  }
}

// Launch shape of the plane kernels: blockIdx.y strides over the rows (images or cotangent
// images), the x-blocks over the row's plane of V-channel groups.
dim3 plane_grid(long long rows, long long plane) {
  const int bx = std::max(1, std::min(cdiv_i(plane, 256), 512));
  const int by = (int)std::max(1LL, std::min<long long>(rows, 65535));
  return dim3(bx, by);
}

// ------------------------------------------------------------------------------ forward
template <int V>
__global__ void __launch_bounds__(256)
k_dw_fwd(const float* __restrict__ x, int images, int H, int W, FastDiv fCG, FastDiv fW,
         const float* __restrict__ w, const float* __restrict__ bias, int act, float* __restrict__ hn,
         float* __restrict__ dphi) {
  const int CG = (int)fCG.d, C = CG * V;
  const int plane = H * W * CG;
  const long long img_elems = (long long)H * W * C;
  for (int n = blockIdx.y; n < images; n += gridDim.y) {
    const float* xi = x + (long long)n * img_elems;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int p = (int)fCG.div(q), cg = q - p * CG;
      const int yy = (int)fW.div(p), xx = p - yy * W;
      const int c0 = cg * V;
      double acc[V];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = 0.0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int sy = yy + t / 3 - 1, sx = xx + t % 3 - 1;
        if ((unsigned)sy < (unsigned)H && (unsigned)sx < (unsigned)W) {
          const Vf<V> a = ldv<V>(xi + (long long)(sy * W + sx) * C + c0);
          const Vf<V> b = ldv<V>(w + t * C + c0);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[v] += (double)a.v[v] * (double)b.v[v];
        }
      }
      Vf<V> ho, dv;
#pragma unroll
      for (int v = 0; v < V; ++v)
        act_pair(act, acc[v] + (bias ? (double)bias[c0 + v] : 0.0), ho.v[v], dv.v[v]);
      const long long o = (long long)n * img_elems + (long long)p * C + c0;
      stv<V>(hn + o, ho);
      stv<V>(dphi + o, dv);
    }
  }
}

template <int V>
__global__ void __launch_bounds__(256)
k_scale_fwd(const float* __restrict__ x, int images, int D, FastDiv fCG, const float* __restrict__ w,
            const float* __restrict__ bias, int act, float* __restrict__ hn, float* __restrict__ dphi) {
  const int CG = (int)fCG.d, C = CG * V;
  const int plane = D * CG;
  for (int n = blockIdx.y; n < images; n += gridDim.y) {
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int p = (int)fCG.div(q), c0 = (q - p * CG) * V;
      const long long o = ((long long)n * D + p) * C + c0;
      const Vf<V> a = ldv<V>(x + o);
      const Vf<V> b = ldv<V>(w + c0);
      Vf<V> ho, dv;
#pragma unroll
      for (int v = 0; v < V; ++v)
        act_pair(act, (double)a.v[v] * (double)b.v[v] + (bias ? (double)bias[c0 + v] : 0.0), ho.v[v], dv.v[v]);
      stv<V>(hn + o, ho);
      stv<V>(dphi + o, dv);
    }
  }
}

// output pixel (yo, xo) = mean of input pixels (2yo + i, 2xo + j), summed in fp64 and rounded once
template <int V>
__global__ void __launch_bounds__(256)
k_pool_fwd(const float* __restrict__ x, int images, int Ho, int Wo, FastDiv fCG, FastDiv fWo,
           float* __restrict__ out) {
  const int CG = (int)fCG.d, C = CG * V;
  const int plane = Ho * Wo * CG;
  const int W = 2 * Wo;
  for (int n = blockIdx.y; n < images; n += gridDim.y) {
    const float* xi = x + (long long)n * 4 * Ho * Wo * C;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int p = (int)fCG.div(q), c0 = (q - p * CG) * V;
      const int yo = (int)fWo.div(p), xo = p - yo * Wo;
      const float* base = xi + (long long)(2 * yo * W + 2 * xo) * C + c0;
      const Vf<V> a = ldv<V>(base), b = ldv<V>(base + C);
      const Vf<V> c = ldv<V>(base + (long long)W * C), d = ldv<V>(base + (long long)W * C + C);
      Vf<V> r;
#pragma unroll
      for (int v = 0; v < V; ++v)
        r.v[v] = (float)((((double)a.v[v] + (double)b.v[v]) + ((double)c.v[v] + (double)d.v[v])) * 0.25);
      stv<V>(out + ((long long)n * Ho * Wo + p) * C + c0, r);
    }
  }
}

// ------------------------------------------------------------------------------ backward
// input pixel q receives G at output pixel q - offset(t) through tap t (zero outside the image)
template <int V>
__global__ void __launch_bounds__(256)
k_dw_bwd(const float* __restrict__ G, int rows, int O, int H, int W, FastDiv fCG, FastDiv fW,
         const float* __restrict__ w, const float* __restrict__ dphi, float* __restrict__ out) {
  const int CG = (int)fCG.d, C = CG * V;
  const int plane = H * W * CG;
  const long long img_elems = (long long)H * W * C;
  for (int r = blockIdx.y; r < rows; r += gridDim.y) {
    const float* Gr = G + (long long)r * img_elems;
    const long long dbase = (long long)(r / O) * img_elems;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int p = (int)fCG.div(q), cg = q - p * CG;
      const int yy = (int)fW.div(p), xx = p - yy * W;
      const int c0 = cg * V;
      float acc[V];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = 0.f;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int sy = yy - (t / 3 - 1), sx = xx - (t % 3 - 1);
        if ((unsigned)sy < (unsigned)H && (unsigned)sx < (unsigned)W) {
          const Vf<V> g = ldv<V>(Gr + (long long)(sy * W + sx) * C + c0);
          const Vf<V> b = ldv<V>(w + t * C + c0);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[v] += g.v[v] * b.v[v];
        }
      }
      const long long o = (long long)p * C + c0;
      Vf<V> res;
      if (dphi) {
        const Vf<V> d = ldv<V>(dphi + dbase + o);
#pragma unroll
        for (int v = 0; v < V; ++v) res.v[v] = acc[v] * d.v[v];
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) res.v[v] = acc[v];
      }
      stv<V>(out + (long long)r * img_elems + o, res);
    }
  }
}

template <int V>
__global__ void __launch_bounds__(256)
k_scale_bwd(const float* __restrict__ G, int rows, int O, int D, FastDiv fCG, const float* __restrict__ w,
            const float* __restrict__ dphi, float* __restrict__ out) {
  const int CG = (int)fCG.d, C = CG * V;
  const int plane = D * CG;
  const long long img_elems = (long long)D * C;
  for (int r = blockIdx.y; r < rows; r += gridDim.y) {
    const long long dbase = (long long)(r / O) * img_elems;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int p = (int)fCG.div(q), c0 = (q - p * CG) * V;
      const long long o = (long long)p * C + c0;
      const Vf<V> g = ldv<V>(G + (long long)r * img_elems + o);
      const Vf<V> b = ldv<V>(w + c0);
      Vf<V> res;
#pragma unroll
      for (int v = 0; v < V; ++v) res.v[v] = g.v[v] * b.v[v];
      if (dphi) {
        const Vf<V> d = ldv<V>(dphi + dbase + o);
#pragma unroll
        for (int v = 0; v < V; ++v) res.v[v] *= d.v[v];
      }
      stv<V>(out + (long long)r * img_elems + o, res);
    }
  }
}

// H, W: the pool's input; every input pixel of a 2x2 window receives a quarter of the window's
// cotangent
template <int V>
__global__ void __launch_bounds__(256)
k_pool_bwd(const float* __restrict__ G, int rows, int O, int H, int W, FastDiv fCG, FastDiv fW,
           const float* __restrict__ dphi, float* __restrict__ out) {
  const int CG = (int)fCG.d, C = CG * V;
  const int plane = H * W * CG;
  const int Wo = W / 2;
  const long long img_elems = (long long)H * W * C;
  const long long gimg_elems = img_elems / 4;
  for (int r = blockIdx.y; r < rows; r += gridDim.y) {
    const float* Gr = G + (long long)r * gimg_elems;
    const long long dbase = (long long)(r / O) * img_elems;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int p = (int)fCG.div(q), c0 = (q - p * CG) * V;
      const int yy = (int)fW.div(p), xx = p - yy * W;
      const Vf<V> g = ldv<V>(Gr + (long long)((yy >> 1) * Wo + (xx >> 1)) * C + c0);
      const long long o = (long long)p * C + c0;
      Vf<V> res;
#pragma unroll
      for (int v = 0; v < V; ++v) res.v[v] = g.v[v] * 0.25f;
      if (dphi) {
        const Vf<V> d = ldv<V>(dphi + dbase + o);
#pragma unroll
        for (int v = 0; v < V; ++v) res.v[v] *= d.v[v];
      }
      stv<V>(out + (long long)r * img_elems + o, res);
    }
  }
}

// ------------------------------------------------------------------------------ pixel sums
// One workgroup per row r = img*O + o (grid-stride).  Lanes take V-channel groups (at most 256
// groups per pass) and pixel groups; each lane accumulates NA = TAPS (+1 with a bias) sums over
// its pixels, and the pixel groups' partial sums are added in a fixed order through LDS.
template <int V, int TAPS, bool BIAS>
__global__ void __launch_bounds__(256)
k_pix_wgrad(const float* __restrict__ G, const float* __restrict__ x, int rows, int O, int H, int W,
            FastDiv fW, int C, float* __restrict__ J, long long ldJ, long long off_w, long long off_b) {
  constexpr int NA = TAPS + (BIAS ? 1 : 0);
  __shared__ float red[256 * NA * V];
  const int CG = C / V;
  const int cgb = CG < 256 ? CG : 256;   // channel groups per pass
  const int PG = 256 / cgb;              // pixel groups
  const int tid = threadIdx.x;
  const int lcg = tid % cgb, pg = tid / cgb;
  const int D = H * W;
  const long long img_elems = (long long)D * C;
  for (int r = blockIdx.x; r < rows; r += gridDim.x) {
    const float* Gr = G + (long long)r * img_elems;
    const float* xi = x + (long long)(r / O) * img_elems;
    for (int cg0 = 0; cg0 < CG; cg0 += cgb) {
      const int cg = cg0 + lcg;
      const bool active = pg < PG && cg < CG;
      float acc[NA][V];
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int v = 0; v < V; ++v) acc[a][v] = 0.f;
      if (active) {
        const int c0 = cg * V;
        for (int p = pg; p < D; p += PG) {
          const Vf<V> g = ldv<V>(Gr + (long long)p * C + c0);
          if constexpr (TAPS == 9) {
            const int yy = (int)fW.div(p), xx = p - yy * W;
#pragma unroll
            for (int t = 0; t < 9; ++t) {
              const int sy = yy + t / 3 - 1, sx = xx + t % 3 - 1;
              if ((unsigned)sy < (unsigned)H && (unsigned)sx < (unsigned)W) {
                const Vf<V> a = ldv<V>(xi + (long long)(sy * W + sx) * C + c0);
#pragma unroll
                for (int v = 0; v < V; ++v) acc[t][v] += g.v[v] * a.v[v];
              }
            }
          } else if constexpr (TAPS == 1) {
            const Vf<V> a = ldv<V>(xi + (long long)p * C + c0);
#pragma unroll
            for (int v = 0; v < V; ++v) acc[0][v] += g.v[v] * a.v[v];
          }
          if constexpr (BIAS) {
#pragma unroll
            for (int v = 0; v < V; ++v) acc[TAPS][v] += g.v[v];
          }
        }
      }
      __syncthreads();   // the previous pass's reduction has read `red`
      if (active) {
#pragma unroll
        for (int a = 0; a < NA; ++a)
#pragma unroll
          for (int v = 0; v < V; ++v) red[((pg * NA + a) * cgb + lcg) * V + v] = acc[a][v];
      }
      __syncthreads();
      const int span = cgb * V;   // channels of this pass
      for (int j = tid; j < NA * span; j += 256) {
        const int a = j / span, rem = j - a * span;
        const int c = cg0 * V + rem;
        if (c < C) {
          float sum = 0.f;
          for (int k = 0; k < PG; ++k) sum += red[(k * NA + a) * span + rem];
          const long long col = (a < TAPS) ? off_w + (long long)a * C + c : off_b + c;
          J[(long long)r * ldJ + col] = sum;
        }
      }
    }
  }
}

template <int V, int TAPS, bool BIAS>
hipError_t pix_wgrad_t(hipStream_t s, const float* G, const float* x, int rows, int O, int H, int W, int C,
                       float* J, long long ldJ, long long off_w, long long off_b) {
  const int grid = std::max(1, std::min(rows, 1 << 20));
  k_pix_wgrad<V, TAPS, BIAS><<<dim3(grid), dim3(256), 0, s>>>(G, x, rows, O, H, W, FastDiv((uint32_t)W), C, J,
                                                              ldJ, off_w, off_b);
  return hipGetLastError();
}

template <int V>
hipError_t pix_wgrad_v(hipStream_t s, const float* G, const float* x, int rows, int O, int H, int W, int C,
                       int taps, int bias, float* J, long long ldJ, long long off_w, long long off_b) {
  if (taps == 9)
    return bias ? pix_wgrad_t<V, 9, true>(s, G, x, rows, O, H, W, C, J, ldJ, off_w, off_b)
                : pix_wgrad_t<V, 9, false>(s, G, x, rows, O, H, W, C, J, ldJ, off_w, off_b);
  if (taps == 1)
    return bias ? pix_wgrad_t<V, 1, true>(s, G, x, rows, O, H, W, C, J, ldJ, off_w, off_b)
                : pix_wgrad_t<V, 1, false>(s, G, x, rows, O, H, W, C, J, ldJ, off_w, off_b);
  if (taps == 0 && bias) return pix_wgrad_t<V, 0, true>(s, G, x, rows, O, H, W, C, J, ldJ, off_w, off_b);
  return hipErrorInvalidValue;
}

bool use_vec4(int C, std::initializer_list<const void*> ptrs) {
  if (C % 4 != 0) return false;
  for (const void* p : ptrs)
    if (p && !al16(p)) return false;
  return true;
}

bool plane_fits(long long images, long long plane) {
  return images >= 0 && plane >= 0 && plane < (1LL << 31) && images * plane < (1LL << 40);
}

}  // namespace

// ------------------------------------------------------------------------------ launchers
hipError_t launch_dw_fwd(hipStream_t s, const float* x, int images, int H, int W, int C, const float* w,
                         const float* bias, int act, float* hn, float* dphi) {
  if (!plane_fits(images, (long long)H * W * C)) return hipErrorInvalidValue;
  if (use_vec4(C, {x, w, hn, dphi})) {
    k_dw_fwd<4><<<plane_grid(images, (long long)H * W * C / 4), dim3(256), 0, s>>>(
        x, images, H, W, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)W), w, bias, act, hn, dphi);
  } else {
    k_dw_fwd<1><<<plane_grid(images, (long long)H * W * C), dim3(256), 0, s>>>(
        x, images, H, W, FastDiv((uint32_t)C), FastDiv((uint32_t)W), w, bias, act, hn, dphi);
  }
  return hipGetLastError();
}

hipError_t launch_scale_fwd(hipStream_t s, const float* x, int images, int D, int C, const float* w,
                            const float* bias, int act, float* hn, float* dphi) {
  if (!plane_fits(images, (long long)D * C)) return hipErrorInvalidValue;
  if (use_vec4(C, {x, w, hn, dphi})) {
    k_scale_fwd<4><<<plane_grid(images, (long long)D * C / 4), dim3(256), 0, s>>>(
        x, images, D, FastDiv((uint32_t)(C / 4)), w, bias, act, hn, dphi);
  } else {
    k_scale_fwd<1><<<plane_grid(images, (long long)D * C), dim3(256), 0, s>>>(
        x, images, D, FastDiv((uint32_t)C), w, bias, act, hn, dphi);
  }
  return hipGetLastError();
}

hipError_t launch_pool_fwd(hipStream_t s, const float* x, int images, int H, int W, int C, float* out) {
  if (H % 2 || W % 2 || !plane_fits(images, (long long)H * W * C)) return hipErrorInvalidValue;
  const int Ho = H / 2, Wo = W / 2;
  if (use_vec4(C, {x, out})) {
    k_pool_fwd<4><<<plane_grid(images, (long long)Ho * Wo * C / 4), dim3(256), 0, s>>>(
        x, images, Ho, Wo, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)Wo), out);
  } else {
    k_pool_fwd<1><<<plane_grid(images, (long long)Ho * Wo * C), dim3(256), 0, s>>>(
        x, images, Ho, Wo, FastDiv((uint32_t)C), FastDiv((uint32_t)Wo), out);
  }
  return hipGetLastError();
}

hipError_t launch_dw_bwd(hipStream_t s, const float* G, int images, int O, int H, int W, int C,
                         const float* w, const float* dphi, float* out) {
  const long long rows = (long long)images * O;
  if (rows >= (1LL << 31) || !plane_fits(rows, (long long)H * W * C)) return hipErrorInvalidValue;
  if (use_vec4(C, {G, w, dphi, out})) {
    k_dw_bwd<4><<<plane_grid(rows, (long long)H * W * C / 4), dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)W), w, dphi, out);
  } else {
    k_dw_bwd<1><<<plane_grid(rows, (long long)H * W * C), dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)C), FastDiv((uint32_t)W), w, dphi, out);
  }
  return hipGetLastError();
}

hipError_t launch_scale_bwd(hipStream_t s, const float* G, int images, int O, int D, int C, const float* w,
                            const float* dphi, float* out) {
  const long long rows = (long long)images * O;
  if (rows >= (1LL << 31) || !plane_fits(rows, (long long)D * C)) return hipErrorInvalidValue;
  if (use_vec4(C, {G, w, dphi, out})) {
    k_scale_bwd<4><<<plane_grid(rows, (long long)D * C / 4), dim3(256), 0, s>>>(
        G, (int)rows, O, D, FastDiv((uint32_t)(C / 4)), w, dphi, out);
  } else {
    k_scale_bwd<1><<<plane_grid(rows, (long long)D * C), dim3(256), 0, s>>>(
        G, (int)rows, O, D, FastDiv((uint32_t)C), w, dphi, out);
  }
  return hipGetLastError();
}

hipError_t launch_pool_bwd(hipStream_t s, const float* G, int images, int O, int H, int W, int C,
                           const float* dphi, float* out) {
  const long long rows = (long long)images * O;
  if (H % 2 || W % 2 || rows >= (1LL << 31) || !plane_fits(rows, (long long)H * W * C))
    return hipErrorInvalidValue;
  if (use_vec4(C, {G, dphi, out})) {
    k_pool_bwd<4><<<plane_grid(rows, (long long)H * W * C / 4), dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)W), dphi, out);
  } else {
    k_pool_bwd<1><<<plane_grid(rows, (long long)H * W * C), dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)C), FastDiv((uint32_t)W), dphi, out);
  }
  return hipGetLastError();
}

hipError_t launch_pix_wgrad(hipStream_t s, const float* G, const float* x, int images, int O, int H, int W,
                            int C, int taps, int bias, float* J, long long ldJ, long long off_w,
                            long long off_b) {
  const long long rows = (long long)images * O;
  if (rows >= (1LL << 31) || !plane_fits(rows, (long long)H * W * C)) return hipErrorInvalidValue;
  if (taps != 0 && taps != 1 && taps != 9) return hipErrorInvalidValue;
  if (use_vec4(C, {G, x}))
    return pix_wgrad_v<4>(s, G, x, (int)rows, O, H, W, C, taps, bias, J, ldJ, off_w, off_b);
  return pix_wgrad_v<1>(s, G, x, (int)rows, O, H, W, C, taps, bias, J, ldJ, off_w, off_b);
}

}  // namespace ntk
