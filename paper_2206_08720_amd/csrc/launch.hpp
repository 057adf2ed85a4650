// launch.hpp -- host-side launchers of the NTK kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>

#include <algorithm>

namespace ntk {

constexpr int kMaxLayers = 64;  // parametrised layers a model may have

// Narrow a row or element count formed in 64 bits to the int the kernels take.  ntk_init keeps
// every array the kernels index below 2^31 elements, so this holds for every call on a handle;
// a count that would wrap is reported as a launch error instead of being truncated.
inline bool to_int(long long v, int& out) {
  if (v < 0 || v > 2147483647LL) return false;
  out = (int)v;
  return true;
}

// Timing hook: every launcher brackets its kernel(s) with prof_begin/prof_end.
struct Profiler;
void prof_begin(Profiler* p, hipStream_t s, int cls);
void prof_end(Profiler* p, hipStream_t s, int cls);

enum KernelClass {
  KC_DENSE_FWD = 0,
  KC_DENSE_BWD,
  KC_BWD_SEED,
  KC_GRAM,
  KC_NTK_FCN,
  KC_TRANSPOSE,
  KC_CONV_FWD,
  KC_CONV_BWD,
  KC_CONV_SEED,
  KC_GAP,
  KC_CONV_WGRAD,
  KC_NTK_SPLITK,
  KC_NTK_REDUCE,
  KC_CONV_PAIRSUM,
  KC_COPY,
  KC_NTK_DIAG,
  KC_JC_JACOBIAN,
  KC_VP_ELEMENTWISE,
  KC_STRUCT_FWD,     // depthwise / scale / pool forward
  KC_STRUCT_BWD,     // depthwise / scale / pool backward
  KC_STRUCT_WGRAD,   // depthwise / scale / bias weight-space cotangents (pixel sums)
  KC_COUNT
};
const char* kernel_class_name(int cls);

// ---- fully-connected path ------------------------------------------------------------
// z = h W^T (+ b);  hn = act(z);  dphi = act'(z).  h [M, K], W [N, K], hn/dphi [M, N].
// Small batches split K over fp64 partials in `part` (capacity in doubles; may be null).  With
// seedG, the epilogue also writes the readout cotangents seedG[m, o, c] = seedW[o, c] dphi[m, c]
// for o < seedO.
long long dense_fwd_part_doubles(long long max_rows, long long max_cols);
// whether the forward of M x N outputs runs as one launch of 16 x 16 blocks (the seed then in it)
bool dense_fwd_small_ok(long long M, long long N);
hipError_t launch_dense_fwd(hipStream_t s, const float* h, const float* W, const float* b, int M,
                            int N, int K, int act, float* hn, float* dphi, double* part,
                            long long part_capacity, const float* seedW = nullptr, int seedO = 0,
                            float* seedG = nullptr);
// out[r, c] = (sum_k G[r, k] Wt[c, k]) * dphi[(r / O), c].  G [R, K], Wt [N, K], dphi [R/O, N].
hipError_t launch_dense_bwd(hipStream_t s, const float* G, const float* Wt, const float* dphi,
                            int R, int N, int K, int O, float* out);
// The same product reading W [K, N] itself (out = (G W) * dphi[r / O]), without a transposed
// copy: dense_bwd_w_ok says whether the shape and buffers take this form.
bool dense_bwd_w_ok(const float* G, const float* W, long long R, long long N, long long K);
hipError_t launch_dense_bwd_w(hipStream_t s, const float* G, const float* W, const float* dphi, int R, int N,
                              int K, int O, float* out);
// Pointwise (1x1) convolution backward: rows r = (img*O + o)*D + p of R cotangent pixels,
// out[r, c] = (sum_k G[r, k] Wt[c, k]) * dphi[img*D + p, c]  (dphi null: the identity).
hipError_t launch_pw_bwd(hipStream_t s, const float* G, const float* Wt, const float* dphi, int R, int N,
                         int K, int O, int D, float* out);
// Wt [C, R] = W^T for W [R, C].
hipError_t launch_transpose(hipStream_t s, const float* W, int R, int C, float* Wt);
// Wt[z] = W[z]^T for z < count (each W[z] R[z] x C[z], row-major), in one launch.
struct TransposeBatch {
  const float* W[kMaxLayers];
  float* Wt[kMaxLayers];
  int R[kMaxLayers], C[kMaxLayers];
  int count;
};
hipError_t launch_transpose_batch(hipStream_t s, const TransposeBatch& b);

struct GramBatch {
  const float* h1[kMaxLayers + 1];
  const float* h2[kMaxLayers + 1];
  float* out[kMaxLayers + 1];
  int K[kMaxLayers + 1];
  float beta[kMaxLayers + 1];
  int count;
};
// out_l[n1, n2] = h1_l[n1] . h2_l[n2] + beta_l for every l (rows of h have stride K_l).
// Batches whose 64 x 64 tiles would not fill num_cu compute units run in 16 x 16 blocks.
hipError_t launch_gram(hipStream_t s, const GramBatch& g, int N1, int N2, int num_cu);
// launch_dense_bwd_w and launch_gram together, in one launch where the layer's tiles leave
// compute units idle and the Grams take 16 x 16 blocks.
hipError_t launch_dense_bwd_w_gram(hipStream_t s, const float* G, const float* W, const float* dphi, int R, int N,
                                   int K, int O, float* out, const GramBatch& g, int N1, int N2, int num_cu);
// out[b][n1][n2] = a1[n1 ld + b bs .. + K] . a2[n2 ld + b bs .. + K] for b < batches (rows of
// stride ld floats, batch b at the float offset b bs of each row)
hipError_t launch_gram_strided(hipStream_t s, const float* a1, const float* a2, int N1, int N2, int K,
                               long long ld, long long bs, int batches, float* out);

struct FcnContraction {
  const float* G1[kMaxLayers];    // cotangents of batch 1, [N1*O, K_l]
  const float* G2[kMaxLayers];    // cotangents of batch 2, [N2*O, K_l]
  const float* gram[kMaxLayers];  // [N1, N2] input Gram (+ bias term) of layer l
  int K[kMaxLayers];
  int L;                          // number of hidden layers (summands with a cotangent Gram)
  const float* gram_readout;      // [N1, N2], multiplies delta_{o1 o2}
  float readout_scale;            // factor of the readout summand (O for the output trace)
};
// theta[n1, n2, o1, o2] = sum_l gram_l[n1,n2] (G1_l G2_l^T)[(n1,o1),(n2,o2)]
//                         + readout_scale gram_readout[n1,n2] delta_{o1 o2}.
// symmetric != 0: batch 2 is batch 1; only upper-triangle tiles run and mirror.
// Large problems use a stream-K schedule over num_cu persistent workgroups with a partial
// buffer `part` of ntk_fcn_part_floats(num_cu) floats (part may be null: no stream-K).
long long ntk_fcn_part_floats(int num_cu);
hipError_t launch_ntk_fcn(hipStream_t s, const FcnContraction& c, int N1, int N2, int O,
                          int symmetric, float* theta, int num_cu, float* part);

// ---- output- and batch-axis variants ---------------------------------------------------
struct RowdotBatch {
  const float* a[kMaxLayers + 1];
  const float* b[kMaxLayers + 1];
  float* out[kMaxLayers + 1];
  long long K[kMaxLayers + 1];    // row length = row stride
  float beta[kMaxLayers + 1];
  int count;
};
// out_j[n] = a_j[n] . b_j[n] + beta_j for n < N and every job j.
hipError_t launch_rowdot(hipStream_t s, const RowdotBatch& r, int N);

struct DiagTerms {
  const float* A[kMaxLayers];     // per sample n: the O x K_l block at A_l + n O K_l (traced: 1 x K_l)
  const float* B[kMaxLayers];
  const float* w[kMaxLayers];     // per-sample weight w_l[n]; null = 1
  long long K[kMaxLayers];
  int count;
  const float* readout;           // per-sample readout scalar; null = none
  float readout_scale;
};
// O > 0: theta[n, o1, o2] (+)= sum_l w_l[n] (A_l[n] B_l[n]^T)[o1, o2] + readout_scale readout[n] delta.
// O = 0 (traced): theta[n] (+)= sum_l w_l[n] (A_l[n] . B_l[n]) + readout_scale readout[n].
// accumulate != 0 adds to theta.  `part` (capacity floats, may be null) holds partial products
// of K segments when the samples alone are too few to fill the device.
hipError_t launch_ntk_diag(hipStream_t s, const DiagTerms& t, int N, int O, int accumulate, float* theta,
                           float* part, long long part_capacity);

// ---- Jacobian-contraction baseline -----------------------------------------------------
// One column chunk of a dense layer's explicit Jacobian block (see kernels_jc.hip):
// out [R, cc*d (+cc)] with rows (n, o), Oe rows per sample.  G [R, ldG] is the cotangent of
// the layer output, or null for the readout layer (identity cotangent; only_o >= 0 when the
// rows are the one output only_o).
hipError_t launch_jc_dense(hipStream_t s, const float* G, long long ldG, const float* h, int d, int R,
                           int Oe, int only_o, int c0, int cc, int bias, float* out);

// ---- NTK-vector products ----------------------------------------------------------------
// out[r, c] = (a[r, c] + b[r, c] + bias[c]) * dphi[r, c]; a, bias, dphi may be null.
hipError_t launch_jvp_combine(hipStream_t s, const float* a, const float* b, const float* bias,
                              const float* dphi, int R, int C, float* out);
// dst = [a (na floats); b (nb floats)] (stacking two batches, one launch).
hipError_t launch_stack2(hipStream_t s, const float* a, long long na, const float* b, long long nb,
                         float* dst);
// out[c] = sum_r x[r, c] for x [R, C].
hipError_t launch_colsum(hipStream_t s, const float* x, int R, int C, float* out);
// out [n, D, C] = u[n, c] / D * dphi[n, p, c]  (adjoint of global average pooling, times act').
hipError_t launch_gap_adjoint(hipStream_t s, const float* u, const float* dphi, int n, int D, int C,
                              float* out);

}  // namespace ntk
