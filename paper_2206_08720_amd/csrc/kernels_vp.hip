// kernels_vp.hip -- elementwise steps of the NTK-vector product Theta(X1, X2) v.
//
// Section 3.3 writes the product as a JVP of batch 1 applied to the VJP of batch 2:
//   theta_c = VJP_{x2}(v)  (the weight-space cotangent: v pulled back through batch 2),
//   Theta v = JVP_{x1}(theta_c)  (that weight-space vector pushed forward through batch 1).
// The matrix products of both passes run on the GEMM kernels of the forward/backward passes;
// the kernels here are the elementwise glue: the tangent of a layer's pre-activation and the
// bias part of the weight-space cotangent.
#include "launch.hpp"

namespace ntk {

// out[r, c] = (a[r, c] + b[r, c] + bias[c]) * dphi[r, c]   (a, bias, dphi may be null)
__global__ void __launch_bounds__(256)
k_jvp_combine(const float* __restrict__ a, const float* __restrict__ b, const float* __restrict__ bias,
              const float* __restrict__ dphi, int R, int C, float* __restrict__ out) {
  const long long total = (long long)R * C;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int c = (int)(i % C);
    float v = b[i];
    if (a) v += a[i];
    if (bias) v += bias[c];
    if (dphi) v *= dphi[i];
    out[i] = v;
  }
}

hipError_t launch_jvp_combine(hipStream_t s, const float* a, const float* b, const float* bias,
                              const float* dphi, int R, int C, float* out) {
  const long long total = (long long)R * C;
  if (total <= 0) return hipSuccess;
  const int blocks = (int)std::min<long long>((total + 255) / 256, 8192);
  k_jvp_combine<<<dim3(blocks), dim3(256), 0, s>>>(a, b, bias, dphi, R, C, out);
  return hipGetLastError();
}

// out[c] = sum_r x[r, c], rows in order (one thread per column)
__global__ void __launch_bounds__(256) k_colsum(const float* __restrict__ x, int R, int C, float* __restrict__ out) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  int r = 0;
  for (; r + 4 <= R; r += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[u] += x[(long long)(r + u) * C + c];
  }
  for (; r < R; ++r) acc[0] += x[(long long)r * C + c];
  out[c] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

hipError_t launch_colsum(hipStream_t s, const float* x, int R, int C, float* out) {
  if (C <= 0) return hipSuccess;
  k_colsum<<<dim3((C + 255) / 256), dim3(256), 0, s>>>(x, R, C, out);
  return hipGetLastError();
}

// Cotangent of the last conv pre-activation from the cotangent u [n, C] of the pooled
// features: out[s, p, c] = u[s, c] / D * dphi[s, p, c] (global average pooling spreads u
// evenly over the D pixels; dphi null: the identity).
__global__ void __launch_bounds__(256)
k_gap_adjoint(const float* __restrict__ u, const float* __restrict__ dphi, int n, int D, int C,
              float* __restrict__ out) {
  const long long total = (long long)n * D * C;
  const float inv = 1.f / (float)D;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const int c = (int)(i % C);
    const long long sp = i / C;
    const int smp = (int)(sp / D);
    out[i] = dphi ? u[(long long)smp * C + c] * inv * dphi[i] : u[(long long)smp * C + c] * inv;
  }
}

hipError_t launch_gap_adjoint(hipStream_t s, const float* u, const float* dphi, int n, int D, int C,
                              float* out) {
  const long long total = (long long)n * D * C;
  if (total <= 0) return hipSuccess;
  const int blocks = (int)std::min<long long>((total + 255) / 256, 8192);
  k_gap_adjoint<<<dim3(blocks), dim3(256), 0, s>>>(u, dphi, n, D, C, out);
  return hipGetLastError();
}

// dst = [a (na floats); b (nb floats)], one launch (the stacked batch [X1; X2]); float4 copies
// when every pointer and both counts allow them.
__global__ void __launch_bounds__(256)
k_stack2(const float* __restrict__ a, long long na, const float* __restrict__ b, long long nb, int vec,
         float* __restrict__ dst) {
  const long long stride = (long long)gridDim.x * 256;
  if (vec) {
    const long long qa = na >> 2, qt = (na + nb) >> 2;
    for (long long i = blockIdx.x * 256LL + threadIdx.x; i < qt; i += stride) {
      const float4 v = i < qa ? reinterpret_cast<const float4*>(a)[i] : reinterpret_cast<const float4*>(b)[i - qa];
      reinterpret_cast<float4*>(dst)[i] = v;
    }
  } else {
    for (long long i = blockIdx.x * 256LL + threadIdx.x; i < na + nb; i += stride)
      dst[i] = i < na ? a[i] : b[i - na];
  }
}

hipError_t launch_stack2(hipStream_t s, const float* a, long long na, const float* b, long long nb,
                         float* dst) {
  const long long total = na + nb;
  if (total <= 0) return hipSuccess;
  const int vec = ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
                    reinterpret_cast<uintptr_t>(dst)) & 15) == 0 && na % 4 == 0 && nb % 4 == 0;
  const long long work = vec ? total / 4 : total;
  const int blocks = (int)std::min<long long>((work + 255) / 256, 4096);
  k_stack2<<<dim3(blocks), dim3(256), 0, s>>>(a, na, b, nb, vec, dst);
  return hipGetLastError();
}

}  // namespace ntk
