// launch_conv.hpp -- host-side launchers of the convolutional NTK kernels (internal).
#pragma once
#include <hip/hip_runtime.h>

#include "launch.hpp"

namespace ntk {

// hn/dphi [images, H, W, Cout] = act / act' of the SAME 3x3 convolution of x [images, H, W, Cin]
// with K [Cout, 3, 3, Cin], plus bias [Cout] when not null (fp64 accumulation).
hipError_t launch_conv_fwd(hipStream_t s, const float* x, int images, int H, int W, int Cin,
                           const float* K, int Cout, int act, const float* bias, float* hn, float* dphi);
// g [images, C] = mean over the D pixels of h [images, D, C].
hipError_t launch_gap(hipStream_t s, const float* h, int images, int D, int C, float* g);
// G [images*O, D, C] = Wd[o, c] / D * dphi[img, p, c]  (dphi null: the identity).
hipError_t launch_conv_seed(hipStream_t s, const float* Wd, const float* dphi, int images, int O,
                            int D, int C, float* G);
// Kt [Cin, 3, 3, Cout] = K [Cout, 2-kh, 2-kw, Cin]  (the kernel of the transposed convolution).
hipError_t launch_conv_flip(hipStream_t s, const float* K, int Cout, int Cin, float* Kt);
// The same for several layers in one launch: Kt_z [Cin_z, T_z, Cout_z] = K_z [Cout_z, T_z - 1 - t, Cin_z]
// for z < count, T_z = 9 (a 3x3 kernel flipped) or 1 (a pointwise kernel transposed).
struct FlipBatch {
  const float* K[kMaxLayers];
  float* Kt[kMaxLayers];
  int Cout[kMaxLayers], Cin[kMaxLayers], taps[kMaxLayers];
  int count;
};
hipError_t launch_conv_flip_batch(hipStream_t s, const FlipBatch& b);
// out [images*O, D, Cin] = conv3x3(G [images*O, H, W, Cg], Kt [Cin, 3, 3, Cg]) * dphi [images, D, Cin]
// (dphi null: the identity).
hipError_t launch_conv_bwd(hipStream_t s, const float* G, int images, int O, int H, int W, int Cg,
                           const float* Kt, int Cin, const float* dphi, float* out);
// J[(s*O + o), off + c*9*Cin + k] = sum_p G[s, o, p, c] patch(h)[s, p, k] for every sample s.
hipError_t launch_conv_wgrad(hipStream_t s, const float* G, const float* h, int images, int O, int H,
                             int W, int C, int Cin, float* J, long long ldJ, long long off);
// Pointwise (1x1) form: J[(s*O + o), off + c*Cin + ci] = sum_p G[s, o, p, c] h[s, p, ci].
hipError_t launch_pw_wgrad(hipStream_t s, const float* G, const float* h, int images, int O, int H,
                           int W, int C, int Cin, float* J, long long ldJ, long long off);
// The same products for Cin % 4 != 0 on the direct-to-LDS path: h [images, H, W, Cin] is first
// copied into xp [images, H, W, Cp] (Cp = Cin rounded up to 4, zero channels past Cin; caller's
// buffer), and the zero columns are not stored.  conv_wgrad_pad_ok: whether the shapes and
// pointers allow it (else the register-staged form of launch_conv_wgrad / launch_pw_wgrad).
bool conv_wgrad_pad_ok(int images, int O, int H, int W, int C, int Cin, const float* G, const float* xp);
hipError_t launch_conv_wgrad_padded(hipStream_t s, const float* G, const float* h, float* xp, int images, int O,
                                    int H, int W, int C, int Cin, float* J, long long ldJ, long long off, bool pw);
// theta[n1, n2, o1, o2] += scale sum_c Wr[o1, c] Wr[o2, c] Mc[c, n1, n2] (Wr [O, C], Mc [C, N1, N2]).
hipError_t launch_readout_fold(hipStream_t s, const float* Wr, int C, int O, const float* Mc, int N1, int N2,
                               float scale, float* theta);
// The same for the traced output theta [N1, N2]: theta += scale sum_c (sum_o Wr[o, c]^2) Mc[c].
hipError_t launch_readout_fold_trace(hipStream_t s, const float* Wr, int C, int O, const float* Mc, int N1, int N2,
                                     float scale, float* theta);
// Mc[c][i] = A1[i, c, :] . A2[i, c, :] for i < n (rows of KC floats at (i C + c) KC): the per-channel
// Grams of the folded last convolution on the batch diagonal (then launch_readout_fold with N1 = n,
// N2 = 1 adds them into theta [n, O, O], launch_readout_fold_trace into theta [n]).
hipError_t launch_fold_rowdot(hipStream_t s, const float* A1, const float* A2, int n, int C, int KC, float* Mc);
// Deterministic split-K product J1 J2^T: plan, partial products, reduction into theta.
int splitk_tile();
// splits * R1 * R2 <= part_capacity (floats) always holds for the returned plan.
int splitk_plan(int R1, int R2, long long K, int symmetric, long long part_capacity, int* chunk_out);
hipError_t launch_ntk_splitk(hipStream_t s, const float* J1, const float* J2, int R1, int R2,
                             long long K, long long ld, int symmetric, int chunk, int splits,
                             float* part);
// accumulate = 0: theta = w (.) partial sum + rscale * readout summand; 1: theta += w (.) partial
// sum.  w [N1, N2] may be null (= 1); gram [N1, N2] may be null (no readout summand).
hipError_t launch_ntk_reduce(hipStream_t s, const float* part, int splits, int N1, int N2, int O,
                             int symmetric, const float* w, const float* gram, float rscale,
                             int accumulate, float* theta);

// Inside-out order of one 3x3 (taps = 9) or pointwise (taps = 1) convolution on the matrix cores
// (see kernels_pairsum.hip): theta (+)= the layer's summand for every input pair, from its input
// h [M, D, Cin] and output cotangent G [M*O, D, C] of the stacked batch (batch 2 from row
// n2_offset).  Gt is a workspace of pairsum_gt_floats(rows of the stacked batch, O, D, C) floats.
// trace != 0: one value per pair, sum_o Theta[o, o] (readout summand O (g1 . g2)).
// diag != 0: only the pairs (n, n), n < n1 = n2; gram is then the per-sample vector g1[n] . g2[n]
// and theta is [n1, ...].  accumulate = 0 writes theta with the readout summand added.
int pairsum_supported(int D);
long long pairsum_gt_floats(long long images, int O, int D, int C);
hipError_t launch_conv_pairsum(hipStream_t s, const float* h, const float* G, float* Gt, int n1, int n2,
                               int n2_offset, int O, int H, int W, int Cin, int C, int taps,
                               const float* gram, int accumulate, int trace, int diag, float* theta);

}  // namespace ntk
