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
#include <type_traits>

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

// Work items q < plane of `rows` planes (images, or cotangent images r = img*per + o), visited
// as f(r, q).  Each workgroup step takes one 256-item chunk of one plane, assigned by
// xcd_sample_tile with the `per` planes of one image as a sample: all chunks of an image -- whose
// 3x3 windows overlap by a row at the chunk edges, and whose O cotangent images share the
// image's act' -- run on one XCD and meet in its L2.  The grid is a multiple of 8 workgroups, so
// a workgroup stays on its XCD across steps.
template <class F>
__device__ __forceinline__ void for_plane_items(int rows, int per, int plane, int ids, F&& f) {
  const int chunks = (plane + 255) / 256, tiles = per * chunks;
  for (int id = blockIdx.x; id < ids; id += gridDim.x) {
    int g, t;
    if (!xcd_sample_tile(id, tiles, rows / per, g, t)) continue;
    const int k = t / chunks;
    const int q = (t - k * chunks) * 256 + (int)threadIdx.x;
    if (q < plane) f(g * per + k, q);
  }
}

// Launch shape of for_plane_items; ids = 0 (nothing launched: an invalid-value error) when the
// chunk ids would not fit an int, which takes more than 2^39 work items.
struct PlaneLaunch {
  dim3 grid;
  int ids;
};
PlaneLaunch plane_launch(long long rows, int per, long long plane) {
  const long long chunks = (plane + 255) / 256, groups = rows / per;
  const long long ids = 8 * ((groups + 7) / 8) * per * chunks;
  if (per <= 0 || rows % per != 0 || ids <= 0 || ids >= (1LL << 31)) return {dim3(1), 0};
  return {dim3((unsigned)std::min<long long>(ids, 1LL << 20)), (int)ids};
}

// ------------------------------------------------------------------------------ 3x3 windows
// Forward (fp64 sums, whose widened window would not fit a taller block in registers): a lane
// computes XS consecutive output pixels of one image row for V channels:
//   acc[j] = sum_{kh, kw} src(y + kh - 1, x0 + j + kw - 1) * tap[kh*3 + kw]   (zero outside).
// The 3 x (XS + 2) input pixels the outputs share are loaded first, all at once (each load
// from a clamped, valid address, the value zeroed outside the image, so no load waits behind a
// branch), then the XS outputs are formed: 3 (XS + 2) loads instead of 9 XS.
template <int V, int XS, typename A>
__device__ __forceinline__ void dw_segment(const float* __restrict__ img, int H, int W, int C, int c0, int y,
                                           int x0, const Vf<V> (&tap)[9], A (&acc)[XS][V]) {
  Vf<V> win[3][XS + 2];
#pragma unroll
  for (int kh = 0; kh < 3; ++kh) {
    const int sy = y + kh - 1;
    const int syc = min(max(sy, 0), H - 1);
#pragma unroll
    for (int j = 0; j < XS + 2; ++j) {
      const int xc = x0 + j - 1;
      const bool ok = (unsigned)sy < (unsigned)H && (unsigned)xc < (unsigned)W;
      const int xcc = min(max(xc, 0), W - 1);
      const Vf<V> t = ldv<V>(img + ((long long)syc * W + xcc) * C + c0);
#pragma unroll
      for (int v = 0; v < V; ++v) win[kh][j].v[v] = ok ? t.v[v] : 0.f;
    }
  }
#pragma unroll
  for (int j = 0; j < XS; ++j) {
#pragma unroll
    for (int v = 0; v < V; ++v) {
      A sum = 0;
#pragma unroll
      for (int kh = 0; kh < 3; ++kh)
#pragma unroll
        for (int kw = 0; kw < 3; ++kw) sum += (A)win[kh][j + kw].v[v] * (A)tap[kh * 3 + kw].v[v];
      acc[j][v] = sum;
    }
  }
}

// Backward (fp32 sums): a lane computes an RS x XS block of output pixels (rows y0 .. y0 + RS - 1,
// columns x0 .. x0 + XS - 1) for V channels, walking down the rows:
//   acc[j] = sum_{kh, kw} src(y + kh - 1, x0 + j + kw - 1) * tap[kh*3 + kw]   (zero outside).
// Three input rows of XS + 2 pixels stay in registers as a ring; each output row loads one new
// input row (issued before the row before is formed), so the block costs (RS + 2)(XS + 2)
// loads instead of 3 (XS + 2) per row.  Every load reads a clamped, valid address and the value
// is zeroed outside the image, so no load waits behind a branch.  emit(y, acc) receives each
// output row inside the image.
template <int V, int XS>
__device__ __forceinline__ void dw_load_row(const float* __restrict__ img, int H, int W, int C, int c0, int sy,
                                            int x0, Vf<V> (&row)[XS + 2]) {
  const int syc = min(max(sy, 0), H - 1);
  const bool rok = (unsigned)sy < (unsigned)H;
#pragma unroll
  for (int j = 0; j < XS + 2; ++j) {
    const int xc = x0 + j - 1;
    const bool ok = rok && (unsigned)xc < (unsigned)W;
    const Vf<V> t = ldv<V>(img + ((long long)syc * W + min(max(xc, 0), W - 1)) * C + c0);
#pragma unroll
    for (int v = 0; v < V; ++v) row[j].v[v] = ok ? t.v[v] : 0.f;
  }
}

template <int V, int XS, int RS, typename A, class Emit>
__device__ __forceinline__ void dw_rows(const float* __restrict__ img, int H, int W, int C, int c0, int y0,
                                        int x0, const Vf<V> (&tap)[9], Emit&& emit) {
  Vf<V> win[3][XS + 2];
  dw_load_row<V, XS>(img, H, W, C, c0, y0 - 1, x0, win[0]);
  dw_load_row<V, XS>(img, H, W, C, c0, y0, x0, win[1]);
#pragma unroll
  for (int i = 0; i < RS; ++i) {
    // ring slots of input rows y - 1, y, y + 1 for output row y = y0 + i
    const int y = y0 + i;
    dw_load_row<V, XS>(img, H, W, C, c0, y + 1, x0, win[(i + 2) % 3]);
    if (y < H) {
      A acc[XS][V];
#pragma unroll
      for (int j = 0; j < XS; ++j)
#pragma unroll
        for (int v = 0; v < V; ++v) {
          A sum = 0;
#pragma unroll
          for (int kh = 0; kh < 3; ++kh)
#pragma unroll
            for (int kw = 0; kw < 3; ++kw) sum += (A)win[(i + kh) % 3][j + kw].v[v] * (A)tap[kh * 3 + kw].v[v];
          acc[j][v] = sum;
        }
      emit(y, acc);
    }
  }
}

// ------------------------------------------------------------------------------ forward
// Work item q of an image = ((y * XB + xb) * CG + cg): XS pixels of row y from x0 = xb * XS.
template <int V, int XS>
__global__ void __launch_bounds__(256)
k_dw_fwd(const float* __restrict__ x, int images, int H, int W, FastDiv fCG, FastDiv fXB,
         const float* __restrict__ w, const float* __restrict__ bias, int act, float* __restrict__ hn,
         float* __restrict__ dphi, int ids) {
  const int CG = (int)fCG.d, C = CG * V, XB = (int)fXB.d;
  const int plane = H * XB * CG;
  const long long img_elems = (long long)H * W * C;
  for_plane_items(images, 1, plane, ids, [&](int n, int q) {
    const float* xi = x + (long long)n * img_elems;
    {
      const int rest = (int)fCG.div(q), cg = q - rest * CG;
      const int yy = (int)fXB.div(rest), xb = rest - yy * XB;
      const int c0 = cg * V, x0 = xb * XS;
      Vf<V> tap[9];
#pragma unroll
      for (int t = 0; t < 9; ++t) tap[t] = ldv<V>(w + t * C + c0);
      Vf<V> bv;
      if (bias) {
        bv = ldv<V>(bias + c0);
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) bv.v[v] = 0.f;
      }
      double acc[XS][V];
      dw_segment<V, XS, double>(xi, H, W, C, c0, yy, x0, tap, acc);
#pragma unroll
      for (int j = 0; j < XS; ++j) {
        if (x0 + j < W) {
          Vf<V> ho, dv;
#pragma unroll
          for (int v = 0; v < V; ++v) act_pair(act, acc[j][v] + (double)bv.v[v], ho.v[v], dv.v[v]);
          const long long o = n * img_elems + ((long long)yy * W + x0 + j) * C + c0;
          stv<V>(hn + o, ho);
          stv<V>(dphi + o, dv);
        }
      }
    }
  });
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
// Input pixel q receives G at output pixel q - offset(t) through tap t: the same 3x3 window
// with the taps flipped, tap'[kh*3 + kw] = w[(2 - kh)*3 + (2 - kw)].  Work item q of a cotangent
// image as in the forward: an RS x XS block of pixels.
template <int V, int XS, int RS>
__global__ void __launch_bounds__(256)
k_dw_bwd(const float* __restrict__ G, int rows, int O, int H, int W, FastDiv fCG, FastDiv fXB,
         const float* __restrict__ w, const float* __restrict__ dphi, float* __restrict__ out, int ids) {
  const int CG = (int)fCG.d, C = CG * V, XB = (int)fXB.d;
  const int plane = ((H + RS - 1) / RS) * XB * CG;
  const long long img_elems = (long long)H * W * C;
  for_plane_items(rows, O, plane, ids, [&](int r, int q) {
    const float* Gr = G + (long long)r * img_elems;
    const float* dimg = dphi ? dphi + (long long)(r / O) * img_elems : nullptr;
    const int rest = (int)fCG.div(q), cg = q - rest * CG;
    const int yb = (int)fXB.div(rest), xb = rest - yb * XB;
    const int c0 = cg * V, x0 = xb * XS;
    Vf<V> tap[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) tap[t] = ldv<V>(w + (8 - t) * C + c0);
    dw_rows<V, XS, RS, float>(Gr, H, W, C, c0, yb * RS, x0, tap, [&](int y, const float (&acc)[XS][V]) {
      // act' of the output pixels (clamped column, unused past W)
      Vf<V> d[XS];
      if (dimg) {
#pragma unroll
        for (int j = 0; j < XS; ++j) d[j] = ldv<V>(dimg + ((long long)y * W + min(x0 + j, W - 1)) * C + c0);
      }
#pragma unroll
      for (int j = 0; j < XS; ++j) {
        if (x0 + j < W) {
          Vf<V> res;
#pragma unroll
          for (int v = 0; v < V; ++v) res.v[v] = dimg ? acc[j][v] * d[j].v[v] : acc[j][v];
          stv<V>(out + (long long)r * img_elems + ((long long)y * W + x0 + j) * C + c0, res);
        }
      }
    });
  });
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
// cotangent.  A lane takes one pooled pixel and writes its window.
template <int V>
__global__ void __launch_bounds__(256)
k_pool_bwd(const float* __restrict__ G, int rows, int O, int H, int W, FastDiv fCG, FastDiv fWo,
           const float* __restrict__ dphi, float* __restrict__ out) {
  const int CG = (int)fCG.d, C = CG * V;
  const int Wo = W / 2;
  const int plane = (H / 2) * Wo * CG;
  const long long img_elems = (long long)H * W * C;
  const long long gimg_elems = img_elems / 4;
  for (int r = blockIdx.y; r < rows; r += gridDim.y) {
    const long long dbase = (long long)(r / O) * img_elems;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < plane; q += gridDim.x * 256) {
      const int pq = (int)fCG.div(q), c0 = (q - pq * CG) * V;
      const int yo = (int)fWo.div(pq), xo = pq - yo * Wo;
      const Vf<V> g = ldv<V>(G + (long long)r * gimg_elems + (long long)pq * C + c0);
      long long o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = ((long long)(2 * yo + (i >> 1)) * W + 2 * xo + (i & 1)) * C + c0;
      Vf<V> res[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < V; ++v) res[i].v[v] = g.v[v] * 0.25f;
      if (dphi) {
        Vf<V> d[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) d[i] = ldv<V>(dphi + dbase + o[i]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int v = 0; v < V; ++v) res[i].v[v] *= d[i].v[v];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) stv<V>(out + (long long)r * img_elems + o[i], res[i]);
    }
  }
}

// ------------------------------------------------------------------------------ pixel sums
// Scale and bias columns (TAPS = 1: sum_p G x, and/or the bias sum_p G).  One workgroup per row
// r = img*O + o (grid-stride).  Lanes take V-channel groups (at most 256 groups per pass) and
// pixel groups; each lane accumulates NA = TAPS (+1 with a bias) sums over its pixels, four
// pixels per step with their loads issued together (clamped pixel index, the sums of pixels past
// D masked), and the pixel groups' partial sums are added in a fixed order through LDS.
template <int V, int TAPS, bool BIAS>
__global__ void __launch_bounds__(256)
k_pix_wgrad(const float* __restrict__ G, const float* __restrict__ x, int rows, int O, int D, int C,
            float* __restrict__ J, long long ldJ, long long off_w, long long off_b) {
  static_assert(TAPS == 0 || TAPS == 1, "depthwise columns are formed by k_dw_wgrad");
  constexpr int NA = TAPS + (BIAS ? 1 : 0);
  constexpr int U = 4;
  __shared__ float red[256 * NA * V];
  const int CG = C / V;
  const int cgb = CG < 256 ? CG : 256;   // channel groups per pass
  const int PG = 256 / cgb;              // pixel groups
  const int tid = threadIdx.x;
  const int lcg = tid % cgb, pg = tid / cgb;
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
        for (int p = pg; p < D; p += U * PG) {
          Vf<V> g[U], a[U];
          float m[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int pu = p + u * PG;
            m[u] = pu < D ? 1.f : 0.f;
            const long long o = (long long)min(pu, D - 1) * C + c0;
            g[u] = ldv<V>(Gr + o);
            if constexpr (TAPS == 1) a[u] = ldv<V>(xi + o);
          }
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int v = 0; v < V; ++v) {
              const float gv = g[u].v[v] * m[u];
              if constexpr (TAPS == 1) acc[0][v] += gv * a[u].v[v];
              if constexpr (BIAS) acc[TAPS][v] += gv;
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

// Depthwise form (9 taps, optional bias): the nine shifted input pixels of a pixel are shared
// by the O cotangent rows of its image, so a workgroup takes one image, one band of its pixels
// and 64 channels (lane = channel, wave = pixel group), loads the nine taps once per pixel and
// accumulates them against OB rows (n, o) at a time (OB: the launcher's choice, close to a
// divisor of O, so that passes carry few unused rows).  The four waves' sums are added in a fixed
// order through LDS; with several bands, each band writes its sums to `part` ([band][row][10 C],
// bias last) and k_band_reduce adds the bands in order.
template <int OB, bool BIAS>
__global__ void __launch_bounds__(256)
k_dw_wgrad(const float* __restrict__ G, const float* __restrict__ x, int images, int O, int H, int W,
           FastDiv fW, int C, int bands, int cgroups, float* __restrict__ out, long long ld_out,
           long long off_w, long long off_b, long long band_stride) {
  constexpr int NA = 9 + (BIAS ? 1 : 0);
  __shared__ float red[4][NA][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int D = H * W;
  const int per_band = (D + bands - 1) / bands;
  const long long img_elems = (long long)D * C;
  const int work = images * bands * cgroups;
  for (int wg = blockIdx.x; wg < work; wg += gridDim.x) {
    const int cgi = wg % cgroups, rest = wg / cgroups;
    const int band = rest % bands, n = rest / bands;
    const int cc = min(cgi * 64 + lane, C - 1);   // lanes past C load a valid channel, unused
    const int p0 = band * per_band, p1 = min(D, p0 + per_band);
    const float* xi = x + (long long)n * img_elems;
    for (int o0 = 0; o0 < O; o0 += OB) {
      float acc[OB][NA];
#pragma unroll
      for (int i = 0; i < OB; ++i)
#pragma unroll
        for (int a = 0; a < NA; ++a) acc[i][a] = 0.f;
      for (int p = p0 + wave; p < p1; p += 4) {
        const int yy = (int)fW.div(p), xx = p - yy * W;
        // every load reads a valid address (clamped pixel, clamped row) and is issued without a
        // branch, so the 17 loads of a pixel are in flight together; rows past O accumulate
        // sums that are never stored
        float xt[9], g[OB];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
          const int sy = yy + t / 3 - 1, sx = xx + t % 3 - 1;
          const bool ok = (unsigned)sy < (unsigned)H && (unsigned)sx < (unsigned)W;
          const int syc = min(max(sy, 0), H - 1), sxc = min(max(sx, 0), W - 1);
          const float v = xi[(long long)(syc * W + sxc) * C + cc];
          xt[t] = ok ? v : 0.f;
        }
#pragma unroll
        for (int i = 0; i < OB; ++i)
          g[i] = G[((long long)n * O + min(o0 + i, O - 1)) * img_elems + (long long)p * C + cc];
#pragma unroll
        for (int i = 0; i < OB; ++i) {
#pragma unroll
          for (int t = 0; t < 9; ++t) acc[i][t] += g[i] * xt[t];
          if constexpr (BIAS) acc[i][9] += g[i];
        }
      }
      // rows o0 + i < O only (uniform over the workgroup); fully unrolled so that acc[i] stays in
      // registers
#pragma unroll
      for (int i = 0; i < OB; ++i) {
        if (o0 + i < O) {
          __syncthreads();   // the previous row's sums have been read
#pragma unroll
          for (int a = 0; a < NA; ++a) red[wave][a][lane] = acc[i][a];
          __syncthreads();
          const long long r = (long long)n * O + o0 + i;
          for (int j = threadIdx.x; j < NA * 64; j += 256) {
            const int a = j >> 6, l = j & 63;
            const int c = cgi * 64 + l;
            if (c < C) {
              const float sum = ((red[0][a][l] + red[1][a][l]) + red[2][a][l]) + red[3][a][l];
              const long long col = a < 9 ? off_w + (long long)a * C + c : off_b + c;
              out[band * band_stride + r * ld_out + col] = sum;
            }
          }
        }
      }
    }
  }
}

// J[r, off_w + j] (j < 9 C) and J[r, off_b + j - 9 C] (the bias, 9 C <= j < ncols) = sum over the
// bands of part[band][r][j] (row stride 10 C), in band order.
__global__ void __launch_bounds__(256)
k_band_reduce(const float* __restrict__ part, int bands, long long rows, int ncols, int C,
              float* __restrict__ J, long long ldJ, long long off_w, long long off_b) {
  const long long total = rows * ncols, band_stride = rows * 10LL * C;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const long long r = i / ncols;
    const int j = (int)(i - r * ncols);
    const long long src = r * 10LL * C + j;
    float sum = 0.f;
    for (int b = 0; b < bands; ++b) sum += part[b * band_stride + src];
    J[r * ldJ + (j < 9 * C ? off_w + j : off_b + (j - 9 * C))] = sum;
  }
}

template <int V, int TAPS, bool BIAS>
hipError_t pix_wgrad_t(hipStream_t s, const float* G, const float* x, int rows, int O, int D, int C, float* J,
                       long long ldJ, long long off_w, long long off_b) {
  const int grid = std::max(1, std::min(rows, 1 << 20));
  k_pix_wgrad<V, TAPS, BIAS><<<dim3(grid), dim3(256), 0, s>>>(G, x, rows, O, D, C, J, ldJ, off_w, off_b);
  return hipGetLastError();
}

template <int V>
hipError_t pix_wgrad_v(hipStream_t s, const float* G, const float* x, int rows, int O, int D, int C, int taps,
                       int bias, float* J, long long ldJ, long long off_w, long long off_b) {
  if (taps == 1)
    return bias ? pix_wgrad_t<V, 1, true>(s, G, x, rows, O, D, C, J, ldJ, off_w, off_b)
                : pix_wgrad_t<V, 1, false>(s, G, x, rows, O, D, C, J, ldJ, off_w, off_b);
  if (taps == 0 && bias) return pix_wgrad_t<V, 0, true>(s, G, x, rows, O, D, C, J, ldJ, off_w, off_b);
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
// output pixels per lane of the depthwise forward (fp64 sums, one row) and output block per
// lane of the backward (fp32: XS pixels of RS rows)
constexpr int kDwFwdXS = 4, kDwBwdXS = 4, kDwBwdRS = 8;

hipError_t launch_dw_fwd(hipStream_t s, const float* x, int images, int H, int W, int C, const float* w,
                         const float* bias, int act, float* hn, float* dphi) {
  if (!plane_fits(images, (long long)H * W * C)) return hipErrorInvalidValue;
  if (images == 0 || H * W * C == 0) return hipSuccess;
  const int XB = cdiv_i(W, kDwFwdXS);
  if (use_vec4(C, {x, w, hn, dphi})) {
    const PlaneLaunch L = plane_launch(images, 1, (long long)H * XB * C / 4);
    if (L.ids == 0) return hipErrorInvalidValue;
    k_dw_fwd<4, kDwFwdXS><<<L.grid, dim3(256), 0, s>>>(
        x, images, H, W, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)XB), w, bias, act, hn, dphi, L.ids);
  } else {
    const PlaneLaunch L = plane_launch(images, 1, (long long)H * XB * C);
    if (L.ids == 0) return hipErrorInvalidValue;
    k_dw_fwd<1, kDwFwdXS><<<L.grid, dim3(256), 0, s>>>(
        x, images, H, W, FastDiv((uint32_t)C), FastDiv((uint32_t)XB), w, bias, act, hn, dphi, L.ids);
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
  if (rows == 0 || H * W * C == 0) return hipSuccess;
  const int XB = cdiv_i(W, kDwBwdXS), YB = cdiv_i(H, kDwBwdRS);
  if (use_vec4(C, {G, w, dphi, out})) {
    const PlaneLaunch L = plane_launch(rows, O, (long long)YB * XB * C / 4);
    if (L.ids == 0) return hipErrorInvalidValue;
    k_dw_bwd<4, kDwBwdXS, kDwBwdRS><<<L.grid, dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)XB), w, dphi, out, L.ids);
  } else {
    const PlaneLaunch L = plane_launch(rows, O, (long long)YB * XB * C);
    if (L.ids == 0) return hipErrorInvalidValue;
    k_dw_bwd<1, kDwBwdXS, kDwBwdRS><<<L.grid, dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)C), FastDiv((uint32_t)XB), w, dphi, out, L.ids);
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
  const long long pooled = (long long)(H / 2) * (W / 2) * C;
  if (use_vec4(C, {G, dphi, out})) {
    k_pool_bwd<4><<<plane_grid(rows, pooled / 4), dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)(C / 4)), FastDiv((uint32_t)(W / 2)), dphi, out);
  } else {
    k_pool_bwd<1><<<plane_grid(rows, pooled), dim3(256), 0, s>>>(
        G, (int)rows, O, H, W, FastDiv((uint32_t)C), FastDiv((uint32_t)(W / 2)), dphi, out);
  }
  return hipGetLastError();
}

hipError_t launch_pix_wgrad(hipStream_t s, const float* G, const float* x, int images, int O, int H, int W,
                            int C, int taps, int bias, float* J, long long ldJ, long long off_w,
                            long long off_b, float* part, long long part_capacity) {
  const long long rows = (long long)images * O;
  if (rows >= (1LL << 31) || !plane_fits(rows, (long long)H * W * C)) return hipErrorInvalidValue;
  if (taps != 0 && taps != 1 && taps != 9) return hipErrorInvalidValue;
  if (taps == 9) {
    // bands of pixels: about four workgroups per compute unit of 256, at least 64 pixels a
    // band, and as many bands' sums as `part` holds
    const int D = H * W, cgroups = cdiv_i(C, 64);
    const long long ncols = 10LL * C;
    const long long per_band = rows * ncols;
    long long bands = std::min<long long>(cdiv_i(1024, (long long)images * cgroups), std::max(1, D / 64));
    if (part && per_band > 0) bands = std::min(bands, part_capacity / per_band);
    else bands = 1;
    bands = std::max(1LL, bands);
    const long long work = (long long)images * bands * cgroups;
    if (work >= (1LL << 31)) return hipErrorInvalidValue;
    const int grid = (int)std::min<long long>(work, 1 << 20);
    float* out = bands > 1 ? part : J;
    const long long ld_out = bands > 1 ? ncols : ldJ;
    const long long ow = bands > 1 ? 0 : off_w, ob = bands > 1 ? 9LL * C : off_b;
    auto go = [&](auto ob_tag) {
      constexpr int OB = decltype(ob_tag)::value;
      if (bias)
        k_dw_wgrad<OB, true><<<dim3(grid), dim3(256), 0, s>>>(G, x, images, O, H, W, FastDiv((uint32_t)W), C,
                                                              (int)bands, cgroups, out, ld_out, ow, ob, per_band);
      else
        k_dw_wgrad<OB, false><<<dim3(grid), dim3(256), 0, s>>>(G, x, images, O, H, W, FastDiv((uint32_t)W), C,
                                                               (int)bands, cgroups, out, ld_out, ow, ob, per_band);
    };
    // cotangent rows per pass: O rounded up to 1, 2, 4, 5 or 8; two passes of 5 for 9 or 10 rows
    // (ten rows' sums in registers make the compiler wait after each load); 8 beyond
    if (O <= 1) go(std::integral_constant<int, 1>{});
    else if (O <= 2) go(std::integral_constant<int, 2>{});
    else if (O <= 4) go(std::integral_constant<int, 4>{});
    else if (O <= 5 || O == 9 || O == 10) go(std::integral_constant<int, 5>{});
    else go(std::integral_constant<int, 8>{});
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || bands == 1) return e;
    // the band sums have a row stride of 10 C; without a bias only the first 9 C are written
    const int nc = (int)(bias ? ncols : 9LL * C);
    const long long total = rows * nc;
    const int rg = (int)std::max(1LL, std::min<long long>((total + 255) / 256, 1 << 16));
    k_band_reduce<<<dim3(rg), dim3(256), 0, s>>>(part, (int)bands, rows, nc, C, J, ldJ, off_w, off_b);
    return hipGetLastError();
  }
  if (use_vec4(C, {G, x}))
    return pix_wgrad_v<4>(s, G, x, (int)rows, O, H * W, C, taps, bias, J, ldJ, off_w, off_b);
  return pix_wgrad_v<1>(s, G, x, (int)rows, O, H * W, C, taps, bias, J, ldJ, off_w, off_b);
}

}  // namespace ntk
