// launch_struct.hpp -- host-side launchers of the kernels for the further structure rules
// (internal): depthwise 3x3 convolutions, per-channel scale layers, biases broadcast over the
// pixels, and 2x2 average pooling.  Activations are NHWC; `images` counts the images of a
// batch, `O` the cotangent images per input image (rows r = img*O + o).  A null `bias` means no
// bias; a null `dphi` means the identity (the layer before has no activation).
#pragma once
#include <hip/hip_runtime.h>

namespace ntk {

// hn/dphi [images, H, W, C] = act / act' of z = depthwise SAME 3x3 cross-correlation of
// x [images, H, W, C] with w [3, 3, C] (+ bias [C]), accumulated in fp64.
hipError_t launch_dw_fwd(hipStream_t s, const float* x, int images, int H, int W, int C, const float* w,
                         const float* bias, int act, float* hn, float* dphi);
// hn/dphi [images, D, C] = act / act' of z = x * w[c] (+ bias[c]) (fp64).
hipError_t launch_scale_fwd(hipStream_t s, const float* x, int images, int D, int C, const float* w,
                            const float* bias, int act, float* hn, float* dphi);
// out [images, H/2, W/2, C] = mean of each 2x2 window of x [images, H, W, C] (H, W even).
hipError_t launch_pool_fwd(hipStream_t s, const float* x, int images, int H, int W, int C, float* out);

// Cotangent of the layer input, times act' of the layer before:
// out [images*O, H, W, C] = (depthwise transposed conv of G [images*O, H, W, C] with w) * dphi[img]
hipError_t launch_dw_bwd(hipStream_t s, const float* G, int images, int O, int H, int W, int C,
                         const float* w, const float* dphi, float* out);
// out [images*O, D, C] = G * w[c] * dphi[img]
hipError_t launch_scale_bwd(hipStream_t s, const float* G, int images, int O, int D, int C, const float* w,
                            const float* dphi, float* out);
// out [images*O, H, W, C] = G [images*O, H/2, W/2, C] at (y/2, x/2) / 4 * dphi[img]  (H, W: pool input)
hipError_t launch_pool_bwd(hipStream_t s, const float* G, int images, int O, int H, int W, int C,
                           const float* dphi, float* out);

// Weight-space cotangents that are sums over pixels, per row r = img*O + o of G [rows, H, W, C]
// and the layer input x [images, H, W, C]:
//   taps = 9: J[r, off_w + t*C + c] = sum_p G[r, p, c] x[img, p + offset(t), c]   (depthwise;
//             offset(t) = (kh - 1, kw - 1) with zero padding)
//   taps = 1: J[r, off_w + c]       = sum_p G[r, p, c] x[img, p, c]                 (scale)
//   taps = 0: no weight columns
//   bias:     J[r, off_b + c]       = sum_p G[r, p, c]                              (any bias)
// With taps = 9 the pixels are split into bands whose sums go to `part` (capacity in floats;
// may be null: one band) and are then added in band order.
hipError_t launch_pix_wgrad(hipStream_t s, const float* G, const float* x, int images, int O, int H, int W,
                            int C, int taps, int bias, float* J, long long ldJ, long long off_w,
                            long long off_b, float* part, long long part_capacity);

}  // namespace ntk
