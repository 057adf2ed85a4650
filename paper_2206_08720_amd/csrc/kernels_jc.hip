// kernels_jc.hip -- explicit Jacobian blocks for the Jacobian-contraction baseline.
//
// The baseline of Section 3.2 forms the per-sample Jacobians df/dtheta explicitly (from the
// reverse-mode Jacobian: O vector-Jacobian products, Section 3.1.3) and contracts them,
// Theta = J(x1) J(x2)^T, at N1 N2 O^2 P multiply-adds.  For a dense layer z = h W^T + b the
// block of W is J[(n,o), (c,j)] = G[(n,o), c] h[n, j] and the block of b is G[(n,o), c]; for
// the readout layer the cotangent G is the identity row e_o.  The kernel below writes one
// column chunk (output units c0 .. c0+cc) of such a block.
#include <stdint.h>

#include "launch.hpp"

namespace ntk {

// out[r, q], r < R (rows (n, o) with Oe rows per sample), q < cc * d (+ cc bias columns):
//   q < cc d:  g(r, c0 + q / d) * h[r / Oe, q % d]
//   q >= cc d: g(r, c0 + q - cc d)
// g(r, c) = G[r * ldG + c], or, for the readout (G null), 1 if c is the output of row r
// (r % Oe, or `only_o` when one output is kept) else 0.
// Rows are spread over gridDim.y, each thread writes 4 consecutive columns of a row (one
// float4 when `vec`: d and the row length multiples of 4, h and out 16-byte aligned).
__device__ __forceinline__ float jc_g(const float* G, long long ldG, int r, int c, int o_r) {
  return G ? G[(long long)r * ldG + c] : (o_r == c ? 1.f : 0.f);
}

__global__ void __launch_bounds__(256)
k_jc_dense(const float* __restrict__ G, long long ldG, const float* __restrict__ h, int d, int R, int Oe,
           int only_o, int c0, int cc, int bias, int vec, float* __restrict__ out) {
  const long long main_cols = (long long)cc * d;
  const long long cols = main_cols + (bias ? cc : 0);
  for (int r = blockIdx.y; r < R; r += gridDim.y) {
    const float* hr = h + (long long)(r / Oe) * d;
    const int o_r = only_o >= 0 ? only_o : r % Oe;
    float* orow = out + (long long)r * cols;
    for (long long q0 = (blockIdx.x * 256LL + threadIdx.x) * 4; q0 < cols; q0 += gridDim.x * 1024LL) {
      if (vec && q0 < main_cols) {
        const int cq = (int)(q0 / d), j = (int)(q0 - (long long)cq * d);
        const float g = jc_g(G, ldG, r, c0 + cq, o_r);
        const float4 hv = *reinterpret_cast<const float4*>(hr + j);
        *reinterpret_cast<float4*>(orow + q0) = make_float4(g * hv.x, g * hv.y, g * hv.z, g * hv.w);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const long long q = q0 + k;
          if (q >= cols) break;
          if (q < main_cols) {
            const int cq = (int)(q / d), j = (int)(q - (long long)cq * d);
            orow[q] = jc_g(G, ldG, r, c0 + cq, o_r) * hr[j];
          } else {
            orow[q] = jc_g(G, ldG, r, c0 + (int)(q - main_cols), o_r);
          }
        }
      }
    }
  }
}

hipError_t launch_jc_dense(hipStream_t s, const float* G, long long ldG, const float* h, int d, int R,
                           int Oe, int only_o, int c0, int cc, int bias, float* out) {
  const long long cols = (long long)cc * d + (bias ? cc : 0);
  if (R <= 0 || cols <= 0) return hipSuccess;
  const int gx = (int)std::min<long long>((cols + 1023) / 1024, 64);
  const int gy = std::min(R, 8192);
  const int vec = d % 4 == 0 && cols % 4 == 0 && (reinterpret_cast<uintptr_t>(h) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  k_jc_dense<<<dim3(gx, gy), dim3(256), 0, s>>>(G, ldG, h, d, R, Oe, only_o, c0, cc, bias, vec, out);
  return hipGetLastError();
}

}  // namespace ntk
