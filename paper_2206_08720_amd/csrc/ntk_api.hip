// ntk_api.hip -- the C ABI declared in include/ntk.h: validation, workspace planning and
// the stream-ordered schedule of kernels for one NTK evaluation.
//
// Schedule (structured derivatives, Section 3.4; FCN per-layer formula of Section 4.1):
//   1. forward pass over the stacked batch [X1; X2] keeping h_l and act'(z_l)
//   2. the O one-hot output cotangents pulled back through every layer at once
//      (the reverse-mode Jacobian of Section 3.1.3 without the weight-space cotangents)
//   3. the layer-input Grams, and 4. the fused per-tile contraction summed over layers.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/ntk.h"
#include "launch.hpp"
#include "launch_conv.hpp"
#include "launch_struct.hpp"

namespace ntk {

const char* kernel_class_name(int cls) {
  static const char* names[KC_COUNT] = {
      "dense_fwd", "dense_bwd", "bwd_seed",  "gram",       "ntk_fcn",    "transpose",    "conv_fwd",
      "conv_bwd",  "conv_seed", "gap",       "conv_wgrad", "ntk_splitk", "ntk_reduce", "conv_pairsum",
      "copy",      "ntk_diag",  "jc_jacobian", "vp_elementwise", "struct_fwd", "struct_bwd", "struct_wgrad"};
  return (cls >= 0 && cls < KC_COUNT) ? names[cls] : "?";
}

struct Profiler {
  bool enabled = false;
  struct Pending {
    int cls;
    hipEvent_t a, b;
  };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> pool;
  double total_ms[KC_COUNT] = {};
  long long launches[KC_COUNT] = {};
  hipEvent_t open_ev = nullptr;
  int open_cls = -1;

  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  ~Profiler() {
    for (auto& p : pending) {
      (void)hipEventDestroy(p.a);
      (void)hipEventDestroy(p.b);
    }
    for (auto e : pool) (void)hipEventDestroy(e);
  }
};

void prof_begin(Profiler* p, hipStream_t s, int cls) {
  if (!p || !p->enabled) return;
  p->open_ev = p->get();
  p->open_cls = cls;
  if (p->open_ev) (void)hipEventRecord(p->open_ev, s);
}
void prof_end(Profiler* p, hipStream_t s, int cls) {
  if (!p || !p->enabled || !p->open_ev || p->open_cls != cls) return;
  hipEvent_t b = p->get();
  if (!b) return;
  (void)hipEventRecord(b, s);
  p->pending.push_back({cls, p->open_ev, b});
  p->open_ev = nullptr;
  p->open_cls = -1;
}

}  // namespace ntk

using namespace ntk;

struct ntk_handle {
  std::vector<ntk_layer_desc> layers;
  int in_h = 1, in_w = 1, in_c = 0, out_dim = 0;
  bool cnn = false;
  int max_n1 = 0, max_n2 = 0;
  // lean plan (ntk_compute_static): no stream-K or split-forward partials, the smallest split-K
  // buffer, so that the workspace is only the arrays one evaluation of the full theta needs
  bool lean = false;
  hipStream_t stream = nullptr;
  // a second stream of the library's own for the independent steps (weight transposes during
  // the forward pass, layer-input Grams during the backward), joined back with events
  hipStream_t aux = nullptr;
  hipEvent_t ev_fork = nullptr, ev_tr = nullptr, ev_fwd = nullptr, ev_gram = nullptr;
  hipEvent_t ev_seed = nullptr, ev_bwd = nullptr;   // split backward: seed done, second half done
  int device = 0;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  int opt_symmetric = 1;
  int opt_conv_order = NTK_CONV_ORDER_AUTO;
  int opt_output = NTK_OUTPUT_FULL;
  int opt_logit = 0;
  int opt_batch = NTK_BATCH_FULL;
  int opt_method = NTK_METHOD_STRUCTURED;
  int opt_graph = 0;
  // NTK_OPT_GRAPH: the recorded graph and the arguments it was recorded with
  hipGraphExec_t graph_exec = nullptr;
  std::vector<uintptr_t> graph_key;
  // graphs are recorded and replayed on a stream of the library's own (the caller's stream may
  // be the null stream, which cannot be captured), ordered after/before the caller's stream by
  // two events
  hipStream_t gstream = nullptr;
  hipEvent_t ev_gin = nullptr, ev_gout = nullptr;
  // Jacobian-contraction baseline: explicit Jacobian chunks of both batches and the split-K
  // partials of their product, allocated by the first call that needs them
  char* jc_ws = nullptr;
  size_t jc_side_floats = 0;
  long long jc_part_capacity = 0;
  // NTK-vector products: the weight-space cotangent and the tangents, allocated by the first
  // ntk_vector_product call
  char* vp_ws = nullptr;
  std::vector<size_t> vp_off_tc, vp_off_tcb;    // theta_c of each weight tensor and bias
  size_t vp_off_dT = 0, vp_off_hT = 0, vp_off_t0 = 0, vp_off_t1 = 0, vp_off_ga = 0, vp_off_gb = 0,
         vp_off_WLt = 0;
  size_t vp_off_u = 0, vp_off_ca = 0, vp_off_cb = 0, vp_off_cd = 0, vp_off_gdot = 0;   // CNN
  std::string err;
  Profiler prof;

  // ---- fully-connected plan: dense layers 0..L (L = number of hidden layers)
  int L = 0;
  std::vector<int> dims;          // d_0 .. d_{L+1}
  std::vector<size_t> off_h;      // h_l,    l = 0..L      [Mmax, d_l]
  std::vector<size_t> off_dphi;   // dphi_l, l = 0..L-1    [Mmax, d_{l+1}]
  std::vector<size_t> off_G;      // G_l,    l = 0..L-1    [Mmax*O, d_{l+1}]
  std::vector<size_t> off_Wt;     // Wt_l,   l = 1..L-1    [d_l, d_{l+1}]
  std::vector<size_t> off_gram;   // gram_l, l = 0..L      [max_n1*max_n2]
  std::vector<int> param_index;   // first parameter slot of dense layer l
  int num_cu = 0;                 // compute units of the device (stream-K workgroup count)
  size_t off_skpart = 0;          // stream-K partial tiles of the contraction
  size_t off_fpart = 0;           // fp64 split-K partials of the small-batch forward
  long long fpart_capacity = 0;   // doubles
  size_t off_vpart = 0;           // split-K partials of the one-output variants (trace, logit)
  long long vpart_capacity = 0;

  // ---- convolutional plan: spatial layers 0..nc-1 (3x3 and depthwise 3x3 convolutions, scale
  //      layers, 2x2 average pools), GAP, dense readout
  int nc = 0, H = 0, W = 0, D = 0;  // the input image
  std::vector<int> ch;            // c_0 .. c_nc: channels at each layer boundary
  std::vector<int> bh, bw;        // image height and width at each layer boundary 0..nc
  std::vector<int> wslot, bslot;  // parameter slots of layer l's weight and bias (-1: none)
  int rslot = 0;                  // parameter slot of the readout weight
  std::vector<size_t> off_ch;     // layer inputs h_l, l = 0..nc (nc: the GAP input) [Mmax, bh_l, bw_l, c_l]
  std::vector<size_t> off_cdphi;  // act'(z_l) of parametrised layers [Mmax, bh_{l+1}, bw_{l+1}, c_{l+1}]
  std::vector<size_t> off_Kt;     // flipped 3x3 kernels [c_l, 9, c_{l+1}] and transposed pointwise
                                  // weights [c_l, c_{l+1}] of the layers l >= 1
  std::vector<long long> joff;    // first column of layer l's weight block (then its bias) in J when
                                  // every layer is outside-in (the NTK-vector product's layout)
  long long Ktot = 0;             // columns of J at most: every weight and bias column
  size_t off_g = 0, off_Gping = 0, off_Gpong = 0, off_J = 0, off_gram_r = 0, off_part = 0;
  size_t off_gt = 0;              // the inside-out kernel's copy of a cotangent [M, C, O, Dp]
  size_t off_mc = 0;              // per-channel Grams of the last convolution [C, N1, N2] (0: none)
  size_t off_xpad = 0;            // a convolution input padded to a multiple of 4 channels (0: none)
  long long part_capacity = 0;    // floats of the split-K partial buffer
};

static thread_local std::string g_init_error;

static int fail(ntk_handle* h, int code, const std::string& msg) {
  if (h)
    h->err = msg;
  else
    g_init_error = msg;
  return code;
}

static int hip_fail(ntk_handle* h, hipError_t e, const char* what) {
  return fail(h, NTK_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// ------------------------------------------------------------------------------ validation
static bool is_spatial_kind(int k) {
  return k == NTK_CONV3X3_SAME || k == NTK_CONV1X1 || k == NTK_DWCONV3X3_SAME || k == NTK_SCALE ||
         k == NTK_AVGPOOL2;
}

static int validate(const ntk_model_desc* m, ntk_handle* tmp) {
  if (!m || !m->layers || m->n_layers <= 0) return fail(nullptr, NTK_E_ARG, "null or empty model descriptor");
  if (m->out_dim <= 0) return fail(nullptr, NTK_E_SHAPE, "out_dim must be positive");
  const int n = m->n_layers;
  for (int i = 0; i < n; ++i) {
    const ntk_layer_desc& L = m->layers[i];
    if (L.kind != NTK_DENSE && L.kind != NTK_GAP && !is_spatial_kind(L.kind))
      return fail(nullptr, NTK_E_UNSUPPORTED, "layer " + std::to_string(i) + ": unknown kind");
    if (L.act != NTK_ACT_NONE && L.act != NTK_ACT_RELU && L.act != NTK_ACT_ERF)
      return fail(nullptr, NTK_E_UNSUPPORTED, "layer " + std::to_string(i) + ": unknown activation");
    if (L.kind != NTK_GAP && L.kind != NTK_AVGPOOL2 && (L.in <= 0 || L.out <= 0))
      return fail(nullptr, NTK_E_SHAPE, "layer " + std::to_string(i) + ": in/out must be positive");
  }
  const ntk_layer_desc& last = m->layers[n - 1];
  if (last.kind != NTK_DENSE)
    return fail(nullptr, NTK_E_UNSUPPORTED, "the last layer must be a dense readout");
  if (last.act != NTK_ACT_NONE)
    return fail(nullptr, NTK_E_UNSUPPORTED, "the readout layer must have no activation (f = z_last)");
  if (last.out != m->out_dim) return fail(nullptr, NTK_E_SHAPE, "last layer out != out_dim");

  bool any_conv = false;
  for (int i = 0; i < n; ++i) any_conv |= m->layers[i].kind != NTK_DENSE;
  if (!any_conv) {
    if (m->in_h != 1 || m->in_w != 1)
      return fail(nullptr, NTK_E_SHAPE, "a fully-connected model takes in_h = in_w = 1");
    if (m->layers[0].in != m->in_c) return fail(nullptr, NTK_E_SHAPE, "layer 0 in != in_c");
    for (int i = 0; i + 1 < n; ++i)
      if (m->layers[i].out != m->layers[i + 1].in)
        return fail(nullptr, NTK_E_SHAPE, "layer " + std::to_string(i) + " out != layer " +
                                               std::to_string(i + 1) + " in");
    if (n - 1 > kMaxLayers)
      return fail(nullptr, NTK_E_UNSUPPORTED, "too many hidden layers (max " + std::to_string(kMaxLayers) + ")");
    tmp->cnn = false;
    return NTK_OK;
  }
  // CNN: spatial layers (3x3, pointwise or depthwise 3x3 convolutions, scale layers, 2x2 pools),
  // then gap, then a dense readout
  int i = 0;
  if (m->in_h <= 0 || m->in_w <= 0 || m->in_c <= 0) return fail(nullptr, NTK_E_SHAPE, "bad input shape");
  int c = m->in_c, hh = m->in_h, ww = m->in_w;
  bool any_param = false;
  while (i < n && is_spatial_kind(m->layers[i].kind)) {
    const ntk_layer_desc& L = m->layers[i];
    const std::string at = "layer " + std::to_string(i) + ": ";
    if (L.kind == NTK_AVGPOOL2) {
      if (L.act != NTK_ACT_NONE || L.has_bias)
        return fail(nullptr, NTK_E_UNSUPPORTED, at + "avgpool2 takes no activation and no bias");
      if (hh % 2 || ww % 2) return fail(nullptr, NTK_E_SHAPE, at + "avgpool2 needs an even height and width");
      hh /= 2;
      ww /= 2;
    } else {
      if (L.in != c) return fail(nullptr, NTK_E_SHAPE, at + "in != previous channels");
      if ((L.kind == NTK_DWCONV3X3_SAME || L.kind == NTK_SCALE) && L.out != L.in)
        return fail(nullptr, NTK_E_SHAPE, at + "depthwise and scale layers keep the channel count (out == in)");
      c = L.out;
      any_param = true;
    }
    ++i;
  }
  if (i == 0 || i > kMaxLayers)
    return fail(nullptr, NTK_E_UNSUPPORTED, "a CNN is 1..64 spatial layers, then gap, then a dense readout");
  if (!any_param)
    return fail(nullptr, NTK_E_UNSUPPORTED, "a CNN needs at least one convolution or scale layer before gap");
  if (i != n - 2 || m->layers[i].kind != NTK_GAP)
    return fail(nullptr, NTK_E_UNSUPPORTED, "a CNN is spatial layers, then gap, then one dense readout");
  if (m->layers[i].act != NTK_ACT_NONE) return fail(nullptr, NTK_E_UNSUPPORTED, "gap takes no activation");
  if (last.in != c) return fail(nullptr, NTK_E_SHAPE, "readout in != conv channels");
  if (last.has_bias) return fail(nullptr, NTK_E_UNSUPPORTED, "the CNN readout has no bias");
  tmp->cnn = true;
  return NTK_OK;
}

// ------------------------------------------------------------------------------ index range
// The launchers and kernels form row counts (samples x outputs x pixels), element offsets
// inside one array and tile counts as 32-bit ints.  All of them stay in range when every array a
// kernel indexes -- each workspace array, the inputs, the parameters and theta -- holds fewer
// than 2^31 elements, which ntk_init checks, before any HIP call, for the largest batches the
// handle allows.  Products are saturated, so the check itself cannot overflow.
constexpr long long kMaxElems = (1LL << 31) - 1;
constexpr long long kSat = 1LL << 62;

static long long smul(long long a, long long b) {
  long long r;
  if (a < 0 || b < 0 || __builtin_mul_overflow(a, b, &r) || r > kSat) return kSat;
  return r;
}
static long long smul(std::initializer_list<long long> f) {
  long long r = 1;
  for (long long x : f) r = smul(r, x);
  return r;
}
static long long sadd(long long a, long long b) { return std::min(kSat, a + b); }

// Largest arrays of the plan for batches of at most n1 and n2 samples, as (elements, what).
// Mirrors plan_fcn / plan_cnn (and the lazily allocated Jacobian-contraction and
// NTK-vector-product buffers), but in saturating arithmetic on the raw descriptor.
static int check_index_range(const ntk_handle& t, long long n1, long long n2) {
  const long long O = t.out_dim, M = sadd(n1, n2), T = 128;   // T: the split-K tile (splitk_tile())
  long long worst = 0;
  std::string what;
  auto need = [&](long long elems, const std::string& w) {
    if (elems > worst) {
      worst = elems;
      what = w;
    }
  };
  auto tiles = [&](long long r1, long long r2) { return smul((r1 + T - 1) / T, (r2 + T - 1) / T); };
  need(smul({n1, n2, O, O}), "theta [n1, n2, O, O]");
  const long long in_elems = smul({(long long)t.in_h, t.in_w, t.in_c});
  need(smul(std::max(n1, n2), in_elems), "an input batch");
  const int n = (int)t.layers.size();
  if (!t.cnn) {
    long long dmax = t.layers[0].in;
    for (int l = 0; l < n; ++l) {
      const ntk_layer_desc& L = t.layers[l];
      dmax = std::max<long long>(dmax, L.out);
      need(smul(M, L.in), "layer " + std::to_string(l) + " inputs [n1 + n2, in]");
      need(smul((long long)L.in, L.out), "layer " + std::to_string(l) + " weights");
      need(smul({M, O, (long long)L.out}), "layer " + std::to_string(l) + " cotangents [(n1 + n2) O, out]");
    }
    need(smul(sadd(1024, tiles(n1, n2)), T * T), "split-K partials of one-output variants");
    need(smul({std::max(n1, n2), O, sadd(dmax, 1)}), "Jacobian-contraction rows");
    need(smul(sadd(1024, tiles(smul(n1, O), smul(n2, O))), T * T), "Jacobian-contraction partials");
    need(smul(dmax, std::max(n1, n2)), "NTK-vector-product tangents");
  } else {
    long long hh = t.in_h, ww = t.in_w, c = t.in_c, ktot = 0;
    const int nc = n - 2;
    for (int l = 0; l < nc; ++l) {
      const ntk_layer_desc& L = t.layers[l];
      const long long plane_in = smul({hh, ww, c});
      need(smul(M, plane_in), "layer " + std::to_string(l) + " inputs [n1 + n2, H, W, C]");
      if (L.kind == NTK_AVGPOOL2) {
        hh /= 2;
        ww /= 2;
        continue;
      }
      const long long wcols = L.kind == NTK_CONV3X3_SAME ? smul({9, c, (long long)L.out})
                              : L.kind == NTK_CONV1X1    ? smul(c, L.out)
                              : L.kind == NTK_DWCONV3X3_SAME ? smul(9, L.out)
                                                             : (long long)L.out;
      need(wcols, "layer " + std::to_string(l) + " weights");
      ktot = sadd(ktot, sadd(wcols, L.has_bias ? L.out : 0));
      c = L.out;
      const long long plane_out = smul({hh, ww, c});
      need(smul(M, plane_out), "layer " + std::to_string(l) + " outputs [n1 + n2, H, W, C]");
      need(smul({M, O, plane_out}), "layer " + std::to_string(l) + " cotangents [(n1 + n2) O, H, W, C]");
      if (L.kind == NTK_CONV3X3_SAME || L.kind == NTK_CONV1X1)   // the inside-out copy [M, C, O, Dp]
        need(smul({M, O, c, 16 * ((smul(hh, ww) + 15) / 16)}),
             "layer " + std::to_string(l) + " cotangent copy of the inside-out order");
    }
    need(smul({M, O, ktot}), "weight-space cotangent columns J [(n1 + n2) O, K]");
    need(smul(sadd(1024, tiles(smul(n1, O), smul(n2, O))), T * T), "split-K partials");
    need(smul(c, O), "readout weights");
    need(sadd(ktot, smul(O, c)), "NTK-vector-product weight-space vector");
    need(smul({std::max(n1, n2), O, sadd(c, 1)}), "Jacobian-contraction rows");
  }
  if (worst <= kMaxElems) return NTK_OK;
  return fail(nullptr, NTK_E_UNSUPPORTED,
              what + " would hold " + std::to_string(worst) +
                  " elements; every array the library indexes must stay below 2^31 (compute theta "
                  "in sample blocks instead)");
}

static size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// ------------------------------------------------------------------------------ planning
static void plan_fcn(ntk_handle* h) {
  const int n = (int)h->layers.size();
  h->L = n - 1;
  const int L = h->L;
  h->dims.resize(L + 2);
  h->dims[0] = h->layers[0].in;
  for (int l = 0; l <= L; ++l) h->dims[l + 1] = h->layers[l].out;
  const size_t Mmax = (size_t)h->max_n1 + h->max_n2;
  const size_t O = h->out_dim;
  size_t off = 0;
  auto take = [&](size_t floats) {
    size_t o = off;
    off = align_up(off + floats * 4);
    return o;
  };
  h->off_h.assign(L + 1, 0);
  h->off_dphi.assign(std::max(L, 1), 0);
  h->off_G.assign(std::max(L, 1), 0);
  h->off_Wt.assign(std::max(L, 1), 0);
  h->off_gram.assign(L + 1, 0);
  for (int l = 0; l <= L; ++l) h->off_h[l] = take(Mmax * h->dims[l]);
  for (int l = 0; l < L; ++l) h->off_dphi[l] = take(Mmax * h->dims[l + 1]);
  for (int l = 0; l < L; ++l) h->off_G[l] = take(Mmax * O * h->dims[l + 1]);
  for (int l = 1; l < L; ++l) h->off_Wt[l] = take((size_t)h->dims[l] * h->dims[l + 1]);
  for (int l = 0; l <= L; ++l) h->off_gram[l] = take((size_t)h->max_n1 * h->max_n2);
  if (h->lean) {   // the full theta only: no stream-K, no split forward, no one-output variants
    h->off_skpart = h->off_fpart = h->off_vpart = 0;
    h->fpart_capacity = h->vpart_capacity = 0;
  } else {
    h->off_skpart = take((size_t)ntk_fcn_part_floats(h->num_cu));
    long long dmax = 1;
    for (int d : h->dims) dmax = std::max<long long>(dmax, d);
    h->fpart_capacity = dense_fwd_part_doubles((long long)Mmax, dmax);
    h->off_fpart = take((size_t)h->fpart_capacity * 2);
    const int T = splitk_tile();
    const size_t tiles_max = (size_t)((h->max_n1 + T - 1) / T) * ((h->max_n2 + T - 1) / T);
    h->vpart_capacity = (long long)(1024 + tiles_max) * T * T;   // >= max_n1 * max_n2
    h->off_vpart = take((size_t)h->vpart_capacity);
  }
  h->ws_bytes = off;
  h->param_index.assign(L + 1, 0);
  int p = 0;
  for (int l = 0; l <= L; ++l) {
    h->param_index[l] = p;
    p += 1 + (h->layers[l].has_bias ? 1 : 0);
  }
}

// Columns of a spatial layer's weight block in J: 9 Cin Cout (3x3 convolution, outside-in),
// Cin Cout (pointwise), 9 C (depthwise), C (scale), 0 (pool).
static long long weight_cols(const ntk_layer_desc& L, int cin) {
  switch (L.kind) {
    case NTK_CONV3X3_SAME: return 9LL * cin * L.out;
    case NTK_CONV1X1: return (long long)cin * L.out;
    case NTK_DWCONV3X3_SAME: return 9LL * L.out;
    case NTK_SCALE: return L.out;
    default: return 0;
  }
}

static void plan_cnn(ntk_handle* h) {
  const int n = (int)h->layers.size();
  h->nc = n - 2;
  h->H = h->in_h;
  h->W = h->in_w;
  h->D = h->H * h->W;
  const int nc = h->nc;
  h->ch.assign(nc + 1, 0);
  h->bh.assign(nc + 1, 0);
  h->bw.assign(nc + 1, 0);
  h->ch[0] = h->in_c;
  h->bh[0] = h->in_h;
  h->bw[0] = h->in_w;
  h->wslot.assign(nc, -1);
  h->bslot.assign(nc, -1);
  int slot = 0;
  for (int l = 0; l < nc; ++l) {
    const ntk_layer_desc& L = h->layers[l];
    const bool pool = L.kind == NTK_AVGPOOL2;
    h->bh[l + 1] = pool ? h->bh[l] / 2 : h->bh[l];
    h->bw[l + 1] = pool ? h->bw[l] / 2 : h->bw[l];
    h->ch[l + 1] = pool ? h->ch[l] : L.out;
    if (!pool) {
      h->wslot[l] = slot++;
      if (L.has_bias) h->bslot[l] = slot++;
    }
  }
  h->rslot = slot;
  const size_t Mmax = (size_t)h->max_n1 + h->max_n2;
  const size_t O = h->out_dim;
  size_t off = 0;
  auto take = [&](size_t floats) {
    size_t o = off;
    off = align_up(off + floats * 4);
    return o;
  };
  auto plane = [&](int b) { return (size_t)h->bh[b] * h->bw[b] * h->ch[b]; };
  size_t gmax = 0;   // largest cotangent image: the output of some layer
  for (int b = 1; b <= nc; ++b) gmax = std::max(gmax, plane(b));
  h->off_ch.assign(nc + 1, 0);
  h->off_cdphi.assign(nc, 0);
  h->off_Kt.assign(nc, 0);
  h->joff.assign(nc, 0);
  for (int l = 0; l <= nc; ++l) h->off_ch[l] = take(Mmax * plane(l));
  for (int l = 0; l < nc; ++l)
    if (h->wslot[l] >= 0) h->off_cdphi[l] = take(Mmax * plane(l + 1));
  for (int l = 1; l < nc; ++l)   // flipped 3x3 kernels, transposed pointwise weights
    if (h->layers[l].kind == NTK_CONV3X3_SAME || h->layers[l].kind == NTK_CONV1X1)
      h->off_Kt[l] = take((size_t)(h->layers[l].kind == NTK_CONV1X1 ? 1 : 9) * h->ch[l] * h->ch[l + 1]);
  h->off_g = take(Mmax * h->ch[nc]);
  h->off_Gping = take(Mmax * O * gmax);
  h->off_Gpong = take(Mmax * O * gmax);
  long long kt = 0;
  for (int l = 0; l < nc; ++l) {
    const ntk_layer_desc& L = h->layers[l];
    h->joff[l] = kt;
    kt += weight_cols(L, h->ch[l]) + (L.has_bias ? L.out : 0);
  }
  h->Ktot = kt;
  h->off_J = take(Mmax * O * (size_t)kt + 4);   // + the 16-byte boundary of a folded layer's rows
  h->off_gram_r = take((size_t)h->max_n1 * h->max_n2);
  {   // the inputs of 3x3 and pointwise convolutions with Cin % 4 != 0, padded for the
      // direct-to-LDS weight-space product
    size_t pad = 0;
    for (int l = 0; l < nc; ++l) {
      const int kind = h->layers[l].kind;
      if ((kind == NTK_CONV3X3_SAME || kind == NTK_CONV1X1) && h->ch[l] % 4 != 0)
        pad = std::max(pad, (size_t)h->bh[l] * h->bw[l] * ((h->ch[l] + 3) & ~3));
    }
    if (pad) h->off_xpad = take(Mmax * pad);
  }
  {   // a last 3x3 or pointwise convolution may contract through per-channel Grams (compute_cnn)
    const int kind = nc >= 1 ? h->layers[nc - 1].kind : -1;
    if ((kind == NTK_CONV3X3_SAME || kind == NTK_CONV1X1) && O >= 2)
      h->off_mc = take((size_t)h->ch[nc] * h->max_n1 * h->max_n2);
  }
  {   // the largest cotangent copy of a convolution the inside-out order can take
    long long gt = 0;
    for (int l = 0; l < nc; ++l) {
      const int kind = h->layers[l].kind;
      const int Dl = h->bh[l] * h->bw[l];
      if ((kind == NTK_CONV3X3_SAME || kind == NTK_CONV1X1) && pairsum_supported(Dl))
        gt = std::max(gt, pairsum_gt_floats((long long)Mmax, (int)O, Dl, h->ch[l + 1]));
    }
    h->off_gt = gt ? take((size_t)gt) : 0;
  }
  const int T = splitk_tile();
  const size_t tiles_max = (size_t)((h->max_n1 * O + T - 1) / T) * ((h->max_n2 * O + T - 1) / T);
  // >= R1max * R2max: the split-K plan never holds fewer than one partial product; the lean plan
  // keeps four (split-K up to 4 ways)
  h->part_capacity = h->lean ? 4LL * h->max_n1 * O * h->max_n2 * O : (long long)(1024 + tiles_max) * T * T;
  h->off_part = take((size_t)h->part_capacity);
  h->ws_bytes = off;
}

static void destroy_sync_objects(ntk_handle* h) {
  if (h->aux) (void)hipStreamSynchronize(h->aux);
  for (hipEvent_t* ev : {&h->ev_fork, &h->ev_tr, &h->ev_fwd, &h->ev_gram, &h->ev_seed, &h->ev_bwd}) {
    if (*ev) (void)hipEventDestroy(*ev);
    *ev = nullptr;
  }
  if (h->aux) (void)hipStreamDestroy(h->aux);
  h->aux = nullptr;
}

// ------------------------------------------------------------------------------ C ABI
extern "C" int ntk_init(const ntk_model_desc* model, int max_n1, int max_n2, void* hip_stream,
                        ntk_handle** out) {
  if (!out) return fail(nullptr, NTK_E_ARG, "out is NULL");
  *out = nullptr;
  if (max_n1 <= 0 || max_n2 <= 0) return fail(nullptr, NTK_E_ARG, "max_n1 and max_n2 must be positive");
  ntk_handle tmp;
  int rc = validate(model, &tmp);
  if (rc != NTK_OK) return rc;
  tmp.layers.assign(model->layers, model->layers + model->n_layers);
  tmp.in_h = model->in_h;
  tmp.in_w = model->in_w;
  tmp.in_c = model->in_c;
  tmp.out_dim = model->out_dim;
  rc = check_index_range(tmp, max_n1, max_n2);
  if (rc != NTK_OK) return rc;
  ntk_handle* h = new (std::nothrow) ntk_handle();
  if (!h) return fail(nullptr, NTK_E_OOM, "host allocation failed");
  h->layers.assign(model->layers, model->layers + model->n_layers);
  h->in_h = model->in_h;
  h->in_w = model->in_w;
  h->in_c = model->in_c;
  h->out_dim = model->out_dim;
  h->cnn = tmp.cnn;
  h->max_n1 = max_n1;
  h->max_n2 = max_n2;
  h->stream = (hipStream_t)hip_stream;
  hipError_t e = hipGetDevice(&h->device);
  if (e != hipSuccess) {
    delete h;
    return hip_fail(nullptr, e, "hipGetDevice");
  }
  e = hipDeviceGetAttribute(&h->num_cu, hipDeviceAttributeMultiprocessorCount, h->device);
  if (e != hipSuccess) {
    delete h;
    return hip_fail(nullptr, e, "hipDeviceGetAttribute");
  }
  if (h->cnn)
    plan_cnn(h);
  else
    plan_fcn(h);
  e = hipMalloc((void**)&h->ws, h->ws_bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    size_t bytes = h->ws_bytes;
    delete h;
    return fail(nullptr, NTK_E_OOM, "workspace allocation of " + std::to_string(bytes) + " bytes failed");
  }
  if (hipStreamCreateWithFlags(&h->aux, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->ev_tr, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->ev_fwd, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->ev_gram, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->ev_seed, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->ev_bwd, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    destroy_sync_objects(h);   // run everything on the one stream
  }
  *out = h;
  return NTK_OK;
}


// ------------------------------------------------------------------------------ shared contraction
// theta (+)= the selected variant of A B^T, for row blocks A [n1*Oe, K] and B [n2*Oe, K]
// (rows (n, o), row stride K): the full product through split-K partials in `part`, the
// output trace as rows (n) of Oe*K columns, the batch diagonal per sample.  No readout term.
static hipError_t contract_rows(ntk_handle* h, const float* A, const float* B, int n1, int n2, int Oe,
                                bool trace, bool diag, bool sym, long long K, int accumulate,
                                float* theta, float* part, long long part_capacity) {
  hipStream_t s = h->stream;
  Profiler* P = &h->prof;
  hipError_t e;
  const bool flat = trace || Oe == 1;
  if (diag) {
    DiagTerms t{};
    t.count = 1;
    t.A[0] = A;
    t.B[0] = B;
    t.w[0] = nullptr;
    t.K[0] = flat ? (long long)Oe * K : K;
    t.readout = nullptr;
    t.readout_scale = 0.f;
    prof_begin(P, s, KC_NTK_DIAG);
    e = launch_ntk_diag(s, t, n1, flat ? 0 : Oe, accumulate, theta, part, part_capacity);
    prof_end(P, s, KC_NTK_DIAG);
    return e;
  }
  const int Or = trace ? 1 : Oe;
  const long long Kc = trace ? (long long)Oe * K : K;
  int R1, R2;
  if (!to_int((long long)n1 * Or, R1) || !to_int((long long)n2 * Or, R2)) return hipErrorInvalidValue;
  int chunk = 0;
  const int splits = splitk_plan(R1, R2, Kc, sym ? 1 : 0, part_capacity, &chunk);
  prof_begin(P, s, KC_NTK_SPLITK);
  e = launch_ntk_splitk(s, A, B, R1, R2, Kc, Kc, sym ? 1 : 0, chunk, splits, part);
  prof_end(P, s, KC_NTK_SPLITK);
  if (e != hipSuccess) return e;
  prof_begin(P, s, KC_NTK_REDUCE);
  e = launch_ntk_reduce(s, part, splits, n1, n2, Or, sym ? 1 : 0, nullptr, nullptr, 1.f, accumulate, theta);
  prof_end(P, s, KC_NTK_REDUCE);
  return e;
}

// The Jacobian-contraction buffers: two chunks of explicit Jacobian rows (one per batch) of at
// least one output unit of the widest layer each, and split-K partials of the full product.
static int ensure_jc_workspace(ntk_handle* h) {
  if (h->jc_ws) return NTK_OK;
  const long long O = h->out_dim;
  const long long R = (long long)std::max(h->max_n1, h->max_n2) * O;
  long long widest = 1;
  if (h->cnn)
    widest = h->ch[h->nc] + 1;
  else
    for (int l = 0; l <= h->L; ++l) widest = std::max<long long>(widest, h->dims[l] + 1);
  h->jc_side_floats = (size_t)std::max<long long>(64LL << 20, R * widest);
  const int T = splitk_tile();
  const long long tiles = (long long)((h->max_n1 * O + T - 1) / T) * ((h->max_n2 * O + T - 1) / T);
  h->jc_part_capacity = (1024 + tiles) * T * T;
  const size_t bytes = (2 * align_up(h->jc_side_floats * 4)) + align_up((size_t)h->jc_part_capacity * 4);
  hipError_t e = hipMalloc((void**)&h->jc_ws, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    h->jc_ws = nullptr;
    return fail(h, NTK_E_OOM, "Jacobian-contraction buffers of " + std::to_string(bytes) + " bytes");
  }
  return NTK_OK;
}

// theta (+)= sum over the column chunks of one dense layer's explicit Jacobian block of the
// variant of J1 J2^T.  G1/G2: cotangent rows of the layer output (null for the readout);
// h1/h2: layer inputs [n, d]; `first` says whether theta is still to be written.
static int jc_dense_layer(ntk_handle* h, const float* G1, const float* G2, long long ldG, const float* h1,
                          const float* h2, int d, int units, bool bias, int n1, int n2, int Oe, int only_o,
                          bool trace, bool diag, bool sym, bool& first, float* theta) {
  hipStream_t s = h->stream;
  Profiler* P = &h->prof;
  float* J1 = reinterpret_cast<float*>(h->jc_ws);
  float* J2 = reinterpret_cast<float*>(h->jc_ws + align_up(h->jc_side_floats * 4));
  float* part = reinterpret_cast<float*>(h->jc_ws + 2 * align_up(h->jc_side_floats * 4));
  const long long R = (long long)std::max(n1, n2) * Oe;
  const int cc = (int)std::max<long long>(1, std::min<long long>(units, (long long)h->jc_side_floats / (R * (d + 1))));
  for (int c0 = 0; c0 < units; c0 += cc) {
    const int c = std::min(cc, units - c0);
    const long long K = (long long)c * d + (bias ? c : 0);
    prof_begin(P, s, KC_JC_JACOBIAN);
    hipError_t e = launch_jc_dense(s, G1, ldG, h1, d, n1 * Oe, Oe, only_o, c0, c, bias ? 1 : 0, J1);
    if (e == hipSuccess && !sym)
      e = launch_jc_dense(s, G2, ldG, h2, d, n2 * Oe, Oe, only_o, c0, c, bias ? 1 : 0, J2);
    prof_end(P, s, KC_JC_JACOBIAN);
    if (e != hipSuccess) return hip_fail(h, e, "explicit Jacobian block");
    e = contract_rows(h, J1, sym ? J1 : J2, n1, n2, Oe, trace, diag, sym, K, first ? 0 : 1, theta, part,
                      h->jc_part_capacity);
    if (e != hipSuccess) return hip_fail(h, e, "Jacobian contraction");
    first = false;
  }
  return NTK_OK;
}

// Forward pass of the stacked batch [X1; X2] (or X1 alone when sym) keeping every layer input
// h_l and act'(z_l); *h0 receives the layer-0 input (X1 itself when sym).
// The layers of the forward pass for the rows [r0, r1) of the stacked batch (h0: its layer-0
// input), on stream st; split-K partials (one buffer) only when use_part.
static int fcn_forward_rows(ntk_handle* h, const float* const* params, const float* h0, int r0, int r1,
                            hipStream_t st, bool use_part, const float* seedW = nullptr, int seedO = 0,
                            float* seedG = nullptr) {
  const int L = h->L;
  Profiler* P = &h->prof;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(h->ws + off); };
  // the readout's own output f is not needed
  for (int l = 0; l < L; ++l) {
    const float* W = params[h->param_index[l]];
    const float* b = h->layers[l].has_bias ? params[h->param_index[l] + 1] : nullptr;
    const float* in = (l == 0 ? h0 : F(h->off_h[l])) + (size_t)r0 * h->dims[l];
    prof_begin(P, st, KC_DENSE_FWD);
    hipError_t e = launch_dense_fwd(st, in, W, b, r1 - r0, h->dims[l + 1], h->dims[l], h->layers[l].act,
                                    F(h->off_h[l + 1]) + (size_t)r0 * h->dims[l + 1],
                                    F(h->off_dphi[l]) + (size_t)r0 * h->dims[l + 1],
                                    use_part ? reinterpret_cast<double*>(h->ws + h->off_fpart) : nullptr,
                                    use_part ? h->fpart_capacity : 0, l == L - 1 ? seedW : nullptr, seedO,
                                    l == L - 1 ? seedG : nullptr);
    prof_end(P, st, KC_DENSE_FWD);
    if (e != hipSuccess) return hip_fail(h, e, "dense forward");
  }
  return NTK_OK;
}

// The stacked batch [X1; X2] (X1 alone when sym) into *h0, on the handle's stream.
static int fcn_stack(ntk_handle* h, const float* const* params, const float* X1, int n1, const float* X2,
                     int n2, bool sym, const float** h0) {
  const int L = h->L;
  for (int l = 0; l <= L; ++l) {
    if (!params[h->param_index[l]]) return fail(h, NTK_E_ARG, "null weight pointer");
    if (h->layers[l].has_bias && !params[h->param_index[l] + 1]) return fail(h, NTK_E_ARG, "null bias pointer");
  }
  *h0 = X1;
  if (!sym) {
    const int d0 = h->dims[0];
    float* dst = reinterpret_cast<float*>(h->ws + h->off_h[0]);
    prof_begin(&h->prof, h->stream, KC_COPY);
    hipError_t e = launch_stack2(h->stream, X1, (long long)n1 * d0, X2, (long long)n2 * d0, dst);
    prof_end(&h->prof, h->stream, KC_COPY);
    if (e != hipSuccess) return hip_fail(h, e, "stacking X1/X2");
    *h0 = dst;
  }
  return NTK_OK;
}

// Forward pass of the stacked batch keeping the layer inputs, on the handle's stream.
static int fcn_forward(ntk_handle* h, const float* const* params, const float* X1, int n1,
                       const float* X2, int n2, bool sym, const float** h0, const float* seedW = nullptr,
                       int seedO = 0, float* seedG = nullptr) {
  int rc = fcn_stack(h, params, X1, n1, X2, n2, sym, h0);
  if (rc != NTK_OK) return rc;
  return fcn_forward_rows(h, params, *h0, 0, sym ? n1 : n1 + n2, h->stream, true, seedW, seedO, seedG);
}

// forward FLOPs from which the FCN path puts independent steps on the second stream
constexpr double kAuxStreamMinFlops = 4e9;

static int compute_fcn(ntk_handle* h, const float* const* params, const float* X1, int n1,
                       const float* X2, int n2, float* theta) {
  const int L = h->L;
  const int O = h->out_dim;
  const bool sym = h->opt_symmetric && X1 == X2 && n1 == n2;
  const int M = sym ? n1 : n1 + n2;
  hipStream_t s = h->stream;
  // independent steps go to the library's second stream when it exists and the problem is big
  // enough for the overlap to outweigh the cross-stream synchronisation (an event record and
  // wait cost about 12 us of host time, so below a few GFLOP a single stream is faster)
  double fwd_flops = 0;
  for (int l = 0; l < L; ++l) fwd_flops += 2.0 * M * h->dims[l] * h->dims[l + 1];
  hipStream_t aux = fwd_flops >= kAuxStreamMinFlops ? h->aux : nullptr;
  hipStream_t sa = aux ? aux : s;
  Profiler* P = &h->prof;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(h->ws + off); };
  hipError_t e;
  const bool logit = h->opt_output == NTK_OUTPUT_LOGIT;
  const bool trace = h->opt_output == NTK_OUTPUT_TRACE;
  const bool diag = h->opt_batch == NTK_BATCH_DIAGONAL;
  const bool jc = h->opt_method == NTK_METHOD_JACOBIAN;
  const int Oe = logit ? 1 : O;
  for (int l = 0; l <= L; ++l)
    if (!params[h->param_index[l]]) return fail(h, NTK_E_ARG, "null weight pointer");
  // set below: every backward layer reads W_l itself (K-outer tiles) where the shapes allow, so
  // that no transposed copies are made; with one stream, the Grams in the launch of the first
  // backward layer
  bool bwd_w = false, gram_in_bwd = false;
  auto transposes = [&](hipStream_t st) -> int {
    if (L < 2 || bwd_w) return NTK_OK;
    TransposeBatch tb{};
    tb.count = L - 1;
    for (int l = 1; l < L; ++l) {
      tb.W[l - 1] = params[h->param_index[l]];
      tb.Wt[l - 1] = F(h->off_Wt[l]);
      tb.R[l - 1] = h->dims[l + 1];
      tb.C[l - 1] = h->dims[l];
    }
    prof_begin(P, st, KC_TRANSPOSE);
    hipError_t err = launch_transpose_batch(st, tb);
    prof_end(P, st, KC_TRANSPOSE);
    return err == hipSuccess ? NTK_OK : hip_fail(h, err, "weight transposes");
  };
  const float* h0 = nullptr;
  auto hptr = [&](int l) -> const float* { return l == 0 ? h0 : F(h->off_h[l]); };
  auto H2 = [&](int l) -> const float* { return sym ? hptr(l) : hptr(l) + (size_t)n1 * h->dims[l]; };
  auto gram_batch = [&]() {
    GramBatch gb{};
    gb.count = L + 1;
    for (int l = 0; l <= L; ++l) {
      gb.h1[l] = hptr(l);
      gb.h2[l] = H2(l);
      gb.out[l] = F(h->off_gram[l]);
      gb.K[l] = h->dims[l];
      gb.beta[l] = h->layers[l].has_bias ? 1.0f : 0.0f;
    }
    return gb;
  };
  // layer-input Grams (the x1.x2 scalars; per-sample scalars on the batch diagonal)
  auto grams = [&](hipStream_t st) -> int {
    hipError_t err;
    if (diag) {
      RowdotBatch rb{};
      rb.count = L + 1;
      for (int l = 0; l <= L; ++l) {
        rb.a[l] = hptr(l);
        rb.b[l] = H2(l);
        rb.out[l] = F(h->off_gram[l]);
        rb.K[l] = h->dims[l];
        rb.beta[l] = h->layers[l].has_bias ? 1.0f : 0.0f;
      }
      prof_begin(P, st, KC_GRAM);
      err = launch_rowdot(st, rb, n1);
      prof_end(P, st, KC_GRAM);
      return err == hipSuccess ? NTK_OK : hip_fail(h, err, "diagonal layer-input scalars");
    }
    const GramBatch gb = gram_batch();
    prof_begin(P, st, KC_GRAM);
    err = launch_gram(st, gb, n1, n2, h->num_cu);
    prof_end(P, st, KC_GRAM);
    return err == hipSuccess ? NTK_OK : hip_fail(h, err, "gram");
  };
  // cotangents of the last hidden pre-activation for all O outputs at once (for the one logit o*
  // alone in NTK_OUTPUT_LOGIT: the cotangent rows are then (n) instead of (n, o)): written by the
  // epilogue of the last forward layer, G[n, o, c] = WL[o, c] act'(z[n, c])
  const float* WL = params[h->param_index[L]] + (logit ? (size_t)h->opt_logit * h->dims[L] : 0);
  // one layer of the cotangent backward for the samples [r0, r1)
  auto bwd_layer = [&](hipStream_t st, int l, int r0, int r1) -> hipError_t {
    const size_t K = h->dims[l + 1], N = h->dims[l];
    if (bwd_w && gram_in_bwd && l == L - 1)
      return launch_dense_bwd_w_gram(st, F(h->off_G[l]) + (size_t)r0 * Oe * K, params[h->param_index[l]],
                                     F(h->off_dphi[l - 1]) + (size_t)r0 * N, (r1 - r0) * Oe, N, K, Oe,
                                     F(h->off_G[l - 1]) + (size_t)r0 * Oe * N, gram_batch(), n1, n2, h->num_cu);
    if (bwd_w)
      return launch_dense_bwd_w(st, F(h->off_G[l]) + (size_t)r0 * Oe * K, params[h->param_index[l]],
                                     F(h->off_dphi[l - 1]) + (size_t)r0 * N, (r1 - r0) * Oe, N, K, Oe,
                                     F(h->off_G[l - 1]) + (size_t)r0 * Oe * N);
    return launch_dense_bwd(st, F(h->off_G[l]) + (size_t)r0 * Oe * K, F(h->off_Wt[l]),
                            F(h->off_dphi[l - 1]) + (size_t)r0 * N, (r1 - r0) * Oe, N, K, Oe,
                            F(h->off_G[l - 1]) + (size_t)r0 * Oe * N);
  };
  auto fork = [&](hipEvent_t ev, hipStream_t from, hipStream_t to) -> int {
    hipError_t err = hipEventRecord(ev, from);
    if (err == hipSuccess) err = hipStreamWaitEvent(to, ev, 0);
    return err == hipSuccess ? NTK_OK : hip_fail(h, err, "stream event");
  };
  // The rows (n, o) are independent through the backward, so with a second stream the samples
  // are split in two halves, each a chain of layer GEMMs on its own stream: one half's partial
  // last round of tiles and its launch gaps are filled by the other half's work.  Split only when
  // every layer of a half still fills the chip (at least 2 tiles of 128 x 128 per CU).  The rows
  // are independent through the forward pass and the seed as well, so these are split with the
  // backward (each half's split-K forward, if any, takes its own half of the partial buffer); the
  // per-kernel profiler (one bracket open at a time) keeps the forward on one stream.
  long long min_tiles = -1;
  for (int l = L - 1; l >= 1; --l) {
    const long long t = ((long long)(M / 2) * Oe + 127) / 128 * ((h->dims[l] + 127) / 128);
    min_tiles = min_tiles < 0 ? t : std::min(min_tiles, t);
  }
  const bool split = aux && L >= 2 && M >= 2 && min_tiles >= 2LL * h->num_cu;
  bwd_w = L >= 2;
  for (int l = 1; l < L; ++l)
    bwd_w = bwd_w && dense_bwd_w_ok(F(h->off_G[l]), params[h->param_index[l]], (long long)M * Oe, h->dims[l],
                                      h->dims[l + 1]);
  gram_in_bwd = bwd_w && !aux && !jc && !diag;
  const int MA = split ? M / 2 : M;   // samples on the main stream; the rest on the second
  const bool halves = split && !P->enabled;
  int rc;
  if (halves) {
    // stream s: the forward and backward of samples [0, MA), then the Grams;
    // stream aux: the weight transposes (when the backward cannot read W itself), then the
    // forward and backward of samples [MA, M)
    if ((rc = fcn_stack(h, params, X1, n1, X2, n2, sym, &h0)) != NTK_OK) return rc;
    if ((rc = fork(h->ev_fork, s, aux)) != NTK_OK || (rc = transposes(aux)) != NTK_OK) return rc;
    if ((e = hipEventRecord(h->ev_tr, aux)) != hipSuccess) return hip_fail(h, e, "stream event");
    for (int l = 0; l < L; ++l) {
      // one layer at a time on each stream, so that both streams have work enqueued early
      const float* W = params[h->param_index[l]];
      const float* b = h->layers[l].has_bias ? params[h->param_index[l] + 1] : nullptr;
      for (int half = 0; half < 2; ++half) {
        const int r0 = half ? MA : 0, r1 = half ? M : MA;
        const float* in = (l == 0 ? h0 : F(h->off_h[l])) + (size_t)r0 * h->dims[l];
        const long long cap = h->fpart_capacity / 2;
        double* part = h->fpart_capacity ? reinterpret_cast<double*>(h->ws + h->off_fpart) + half * cap : nullptr;
        const bool last = l == L - 1;
        e = launch_dense_fwd(half ? aux : s, in, W, b, r1 - r0, h->dims[l + 1], h->dims[l], h->layers[l].act,
                             F(h->off_h[l + 1]) + (size_t)r0 * h->dims[l + 1],
                             F(h->off_dphi[l]) + (size_t)r0 * h->dims[l + 1], part, part ? cap : 0,
                             last ? WL : nullptr, Oe, last ? F(h->off_G[l]) + (size_t)r0 * Oe * h->dims[l + 1] : nullptr);
        if (e != hipSuccess) return hip_fail(h, e, "dense forward");
      }
    }
    if ((e = hipEventRecord(h->ev_fwd, aux)) != hipSuccess) return hip_fail(h, e, "stream event");
    if ((e = hipStreamWaitEvent(s, h->ev_tr, 0)) != hipSuccess) return hip_fail(h, e, "stream join");
    for (int l = L - 1; l >= 1; --l) {
      e = bwd_layer(s, l, 0, MA);
      if (e == hipSuccess) e = bwd_layer(aux, l, MA, M);
      if (e != hipSuccess) return hip_fail(h, e, "dense backward");
    }
    if ((e = hipEventRecord(h->ev_bwd, aux)) != hipSuccess) return hip_fail(h, e, "stream event");
    if (!jc) {
      if ((e = hipStreamWaitEvent(s, h->ev_fwd, 0)) != hipSuccess) return hip_fail(h, e, "stream join");
      if ((rc = grams(s)) != NTK_OK) return rc;
    }
    if ((e = hipStreamWaitEvent(s, h->ev_bwd, 0)) != hipSuccess) return hip_fail(h, e, "stream join");
  } else {
    // 0. weight transposes for a backward that cannot read W itself, on the second stream
    //    while the forward runs
    if (aux && (rc = fork(h->ev_fork, s, aux)) != NTK_OK) return rc;
    if ((rc = transposes(sa)) != NTK_OK) return rc;
    if (aux && (e = hipEventRecord(h->ev_tr, sa)) != hipSuccess) return hip_fail(h, e, "stream event");
    // 1. forward pass keeping the layer inputs, and the readout cotangents in the last layer's
    //    epilogue
    if ((rc = L >= 1 ? fcn_forward(h, params, X1, n1, X2, n2, sym, &h0, WL, Oe, F(h->off_G[L - 1]))
                     : fcn_forward(h, params, X1, n1, X2, n2, sym, &h0)) != NTK_OK)
      return rc;
    // 2. the Grams, on the second stream while the backward runs (or in the first backward
    //    layer's launch)
    if (!jc && !gram_in_bwd) {
      if (aux && (rc = fork(h->ev_fwd, s, sa)) != NTK_OK) return rc;
      if ((rc = grams(sa)) != NTK_OK) return rc;
      if (aux && (e = hipEventRecord(h->ev_gram, sa)) != hipSuccess) return hip_fail(h, e, "stream event");
    }
    // 3. the cotangents of every hidden pre-activation
    if (aux && (e = hipStreamWaitEvent(s, h->ev_tr, 0)) != hipSuccess) return hip_fail(h, e, "stream join");
    if (L >= 1) {
      if (split && (rc = fork(h->ev_seed, s, aux)) != NTK_OK) return rc;
      prof_begin(P, s, KC_DENSE_BWD);
      for (int l = L - 1; l >= 1; --l) {
        e = bwd_layer(s, l, 0, MA);
        if (e == hipSuccess && split) e = bwd_layer(aux, l, MA, M);
        if (e != hipSuccess) return hip_fail(h, e, "dense backward");
      }
      if (split && (rc = fork(h->ev_bwd, aux, s)) != NTK_OK) return rc;
      prof_end(P, s, KC_DENSE_BWD);
    }
    if (!jc && aux && (e = hipStreamWaitEvent(s, h->ev_gram, 0)) != hipSuccess)
      return hip_fail(h, e, "stream join");
  }
  auto G1 = [&](int l) -> const float* { return F(h->off_G[l]); };
  auto G2 = [&](int l) -> const float* {
    return sym ? F(h->off_G[l]) : F(h->off_G[l]) + (size_t)n1 * Oe * h->dims[l + 1];
  };
  const float rscale = trace ? (float)O : 1.f;   // sum over o of delta_{oo} for the trace
  if (h->opt_method == NTK_METHOD_JACOBIAN) {
    // Jacobian-contraction baseline: every weight tensor's explicit Jacobian block, chunk by
    // chunk, contracted into theta (the readout's cotangent is the identity)
    int rc = ensure_jc_workspace(h);
    if (rc != NTK_OK) return rc;
    bool first = true;
    const int only_o = logit ? h->opt_logit : -1;
    for (int l = 0; l <= L; ++l) {
      const bool readout = l == L;
      rc = jc_dense_layer(h, readout ? nullptr : G1(l), readout ? nullptr : G2(l), h->dims[l + 1], hptr(l),
                          H2(l), h->dims[l], h->dims[l + 1], h->layers[l].has_bias != 0, n1, n2, Oe, only_o,
                          trace, diag, sym, first, theta);
      if (rc != NTK_OK) return rc;
    }
    return NTK_OK;
  }
  if (diag) {
    // batch diagonal: theta[n] = sum_l d_l[n] G1_l[n] G2_l[n]^T + d_L[n] I with the per-sample
    // layer-input scalars d_l[n] = h1_l[n] . h2_l[n] (+1) (traced: a dot of O*K_l columns)
    DiagTerms t{};
    t.count = L;
    const bool flat = trace || logit;
    for (int l = 0; l < L; ++l) {
      t.A[l] = G1(l);
      t.B[l] = G2(l);
      t.w[l] = F(h->off_gram[l]);
      t.K[l] = (long long)(flat ? Oe : 1) * h->dims[l + 1];
    }
    t.readout = F(h->off_gram[L]);
    t.readout_scale = rscale;
    prof_begin(P, s, KC_NTK_DIAG);
    e = launch_ntk_diag(s, t, n1, flat ? 0 : O, 0, theta, F(h->off_vpart), h->vpart_capacity);
    prof_end(P, s, KC_NTK_DIAG);
    if (e != hipSuccess) return hip_fail(h, e, "diagonal contraction");
    return NTK_OK;
  }
  if (trace || logit) {
    // 4'. one output: per layer a split-K product of the cotangent rows (n) of Oe*K_l columns,
    //     weighted by gram_l and accumulated into theta [n1, n2] layer by layer
    if (L == 0) {
      prof_begin(P, s, KC_NTK_REDUCE);
      e = launch_ntk_reduce(s, F(h->off_vpart), 0, n1, n2, 1, 0, nullptr, F(h->off_gram[L]), rscale, 0,
                            theta);
      prof_end(P, s, KC_NTK_REDUCE);
      if (e != hipSuccess) return hip_fail(h, e, "readout summand");
    }
    for (int l = 0; l < L; ++l) {
      const long long K = (long long)Oe * h->dims[l + 1];
      int chunk = 0;
      const int splits = splitk_plan(n1, n2, K, sym ? 1 : 0, h->vpart_capacity, &chunk);
      prof_begin(P, s, KC_NTK_SPLITK);
      e = launch_ntk_splitk(s, G1(l), G2(l), n1, n2, K, K, sym ? 1 : 0, chunk, splits, F(h->off_vpart));
      prof_end(P, s, KC_NTK_SPLITK);
      if (e != hipSuccess) return hip_fail(h, e, "split-K contraction");
      prof_begin(P, s, KC_NTK_REDUCE);
      e = launch_ntk_reduce(s, F(h->off_vpart), splits, n1, n2, 1, sym ? 1 : 0, F(h->off_gram[l]),
                            F(h->off_gram[L]), rscale, l > 0 ? 1 : 0, theta);
      prof_end(P, s, KC_NTK_REDUCE);
      if (e != hipSuccess) return hip_fail(h, e, "split-K reduction");
    }
    return NTK_OK;
  }
  // 4. fused contraction summed over layers, written as theta[n1][n2][o1][o2]
  FcnContraction c{};
  c.L = L;
  for (int l = 0; l < L; ++l) {
    c.G1[l] = G1(l);
    c.G2[l] = G2(l);
    c.gram[l] = F(h->off_gram[l]);
    c.K[l] = h->dims[l + 1];
  }
  c.gram_readout = F(h->off_gram[L]);
  c.readout_scale = 1.f;
  prof_begin(P, s, KC_NTK_FCN);
  e = launch_ntk_fcn(s, c, n1, n2, O, sym ? 1 : 0, theta, h->num_cu, h->lean ? nullptr : F(h->off_skpart));
  prof_end(P, s, KC_NTK_FCN);
  if (e != hipSuccess) return hip_fail(h, e, "ntk contraction");
  return NTK_OK;
}

// CNN forward pass of the stacked batch [X1; X2] (or X1 alone when sym), keeping every spatial
// layer's input and act'(z_l), then the global average pool g; *h0 receives the layer-0 input.
static int cnn_forward(ntk_handle* h, const float* const* params, const float* X1, int n1,
                       const float* X2, int n2, bool sym, const float** h0) {
  const int nc = h->nc;
  const int M = sym ? n1 : n1 + n2;
  hipStream_t s = h->stream;
  Profiler* P = &h->prof;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(h->ws + off); };
  for (int i = 0; i <= h->rslot; ++i)
    if (!params[i]) return fail(h, NTK_E_ARG, "null parameter pointer");
  hipError_t e;
  const size_t img_floats = (size_t)h->D * h->ch[0];
  *h0 = X1;
  if (!sym) {
    prof_begin(P, s, KC_COPY);
    e = launch_stack2(s, X1, (long long)n1 * img_floats, X2, (long long)n2 * img_floats, F(h->off_ch[0]));
    prof_end(P, s, KC_COPY);
    if (e != hipSuccess) return hip_fail(h, e, "stacking X1/X2");
    *h0 = F(h->off_ch[0]);
  }
  for (int l = 0; l < nc; ++l) {
    const ntk_layer_desc& L = h->layers[l];
    const float* x = l == 0 ? *h0 : F(h->off_ch[l]);
    float* out = F(h->off_ch[l + 1]);
    float* dphi = F(h->off_cdphi[l]);
    const float* w = h->wslot[l] >= 0 ? params[h->wslot[l]] : nullptr;
    const float* b = h->bslot[l] >= 0 ? params[h->bslot[l]] : nullptr;
    const int Hl = h->bh[l], Wl = h->bw[l], C = h->ch[l];
    if (L.kind == NTK_CONV3X3_SAME) {
      prof_begin(P, s, KC_CONV_FWD);
      e = launch_conv_fwd(s, x, M, Hl, Wl, C, w, L.out, L.act, b, out, dphi);
      prof_end(P, s, KC_CONV_FWD);
    } else if (L.kind == NTK_CONV1X1) {   // a dense layer at every pixel
      prof_begin(P, s, KC_CONV_FWD);
      e = launch_dense_fwd(s, x, w, b, M * Hl * Wl, L.out, C, L.act, out, dphi, nullptr, 0);
      prof_end(P, s, KC_CONV_FWD);
    } else {
      prof_begin(P, s, KC_STRUCT_FWD);
      if (L.kind == NTK_DWCONV3X3_SAME)
        e = launch_dw_fwd(s, x, M, Hl, Wl, C, w, b, L.act, out, dphi);
      else if (L.kind == NTK_SCALE)
        e = launch_scale_fwd(s, x, M, Hl * Wl, C, w, b, L.act, out, dphi);
      else
        e = launch_pool_fwd(s, x, M, Hl, Wl, C, out);
      prof_end(P, s, KC_STRUCT_FWD);
    }
    if (e != hipSuccess) return hip_fail(h, e, "forward pass");
  }
  prof_begin(P, s, KC_GAP);
  e = launch_gap(s, F(h->off_ch[nc]), M, h->bh[nc] * h->bw[nc], h->ch[nc], F(h->off_g));
  prof_end(P, s, KC_GAP);
  if (e != hipSuccess) return hip_fail(h, e, "global average pooling");
  return NTK_OK;
}

// The inside-out order's cost for the order choice: the matrix-core work its kernel executes
// (pixels padded to Dp = 16 ceil(D / 16), outputs to 16 ceil(Oe / 16), input channels to 16 per
// step; per block of 16 x 16 outputs the pixel Gram Dp^2 Cin, the product with the patch-pair Gram
// 16 Dp^2 C and the output product 256 Dp C, multiply-adds per input pair), times its measured
// time per multiply-add relative to the outside-in products.
constexpr double kInsideOutTimeWeight = 1.0;

static double inside_out_cost(double pairs, int D, int Cin, int C, int Oe, bool trace) {
  const double Dp = 16.0 * ((D + 15) / 16), Ci = 16.0 * ((Cin + 15) / 16), nob = (Oe + 15) / 16;
  const double gram_blocks = trace ? 1 : nob * nob, out_blocks = trace ? nob : nob * nob;
  return kInsideOutTimeWeight * pairs *
         (gram_blocks * Dp * Dp * Ci + out_blocks * (16.0 * Dp * Dp * C + 256.0 * Dp * C));
}

static int compute_cnn(ntk_handle* h, const float* const* params, const float* X1, int n1,
                       const float* X2, int n2, float* theta) {
  const int nc = h->nc, O = h->out_dim;
  const bool sym = h->opt_symmetric && X1 == X2 && n1 == n2;
  const int M = sym ? n1 : n1 + n2;
  hipStream_t s = h->stream;
  Profiler* P = &h->prof;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(h->ws + off); };
  // variants: one logit (the cotangent rows are then (n) instead of (n, o)), the trace over
  // outputs, the batch diagonal (pairs (n, n) only)
  const bool logit = h->opt_output == NTK_OUTPUT_LOGIT;
  const bool trace = h->opt_output == NTK_OUTPUT_TRACE;
  const bool diag = h->opt_batch == NTK_BATCH_DIAGONAL;
  const int Oe = logit ? 1 : O;
  const double pairs = diag ? (double)n1 : (double)n1 * n2;
  const double Oc = trace ? (double)O : (double)Oe * Oe;   // output pairs per input pair
  // contraction order of each 3x3 (F = 9 taps) or pointwise (F = 1) convolution: the outside-in
  // cost of the appendix "CNN NTK Complexity" (N1 N2 O^2 F Cin Cout plus forming J, N O D F Cin Cout
  // per sample) against the matrix-core work the inside-out kernel executes (inside_out_cost), or
  // the forced option; inside-out only for images of at most 64 pixels.  Depthwise
  // and scale layers (block-diagonal weight-space Jacobians, 9 C and C columns) and every bias
  // (output block-tiled, C columns) always contract outside-in: their O^2 P term is the
  // smallest of the orders there.
  std::vector<char> inside(nc, 0);
  for (int l = 0; l < nc; ++l) {
    const int kind = h->layers[l].kind;
    if ((kind != NTK_CONV3X3_SAME && kind != NTK_CONV1X1) || h->opt_method == NTK_METHOD_JACOBIAN) continue;
    const double F = kind == NTK_CONV1X1 ? 1 : 9;
    const int Dl = h->bh[l] * h->bw[l];
    const bool io_ok = pairsum_supported(Dl) != 0;
    const double Cin = h->ch[l], Co = h->ch[l + 1];
    const double oi = pairs * Oc * F * Cin * Co + (double)M * Oe * Dl * F * Cin * Co;
    const double io = inside_out_cost(pairs, Dl, h->ch[l], h->ch[l + 1], Oe, trace);
    if (h->opt_conv_order == NTK_CONV_ORDER_INSIDE_OUT) {
      if (!io_ok) return fail(h, NTK_E_UNSUPPORTED, "the inside-out order needs images of at most 64 pixels");
      inside[l] = 1;
    } else if (h->opt_conv_order == NTK_CONV_ORDER_AUTO) {
      inside[l] = (io_ok && io < oi) ? 1 : 0;
    }
  }
  // The last convolution's output cotangent is the readout's through the global pool,
  // G[n, o, p, c] = Wr[o, c] act'(z[n, p, c]) / D, so its weight-space columns factor as
  // Wr[o, c] A[n, c, k] / D with A[n, c, k] = sum_p act'(z[n, p, c]) patch[n, p, k], and its
  // summand is sum_c Wr[o1, c] Wr[o2, c] (A1[., c, .] A2[., c, .]^T)[n1, n2] / D^2: the O outputs
  // leave that layer's weight-space product and contraction ("fold").  Outside-in layers only, the
  // full O x O output or its trace (then sum_c (sum_o Wr[o, c]^2) Gram_c / D^2), on the full batch
  // or its diagonal (the per-channel Grams' diagonals), with other columns in J (their contraction
  // then writes theta first).
  const int ll = nc - 1;
  bool fold = nc >= 1 && h->off_mc && h->wslot[ll] >= 0 && O >= 2 && !logit &&
              h->opt_method != NTK_METHOD_JACOBIAN &&
              (h->layers[ll].kind == NTK_CONV3X3_SAME || h->layers[ll].kind == NTK_CONV1X1);
  if (fold) {   // other weight-space columns: a bias, a depthwise or scale layer, an outside-in conv
    bool others = h->layers[ll].has_bias != 0;
    for (int l = 0; l < ll; ++l) {
      const int kind = h->layers[l].kind;
      others = others || h->layers[l].has_bias || kind == NTK_DWCONV3X3_SAME || kind == NTK_SCALE ||
               ((kind == NTK_CONV3X3_SAME || kind == NTK_CONV1X1) && !inside[l]);
    }
    fold = others;
  }
  // With the fold available, the cost model's outside-in cost of the last convolution is that of
  // the fold: the O-free rows M D F Cin Cout, the per-channel Grams N1 N2 F Cin Cout and their
  // O x O sums N1 N2 O^2 Cout.
  if (fold && inside[ll] && h->opt_conv_order == NTK_CONV_ORDER_AUTO) {
    const ntk_layer_desc& L = h->layers[ll];
    const double F = L.kind == NTK_CONV1X1 ? 1 : 9;
    const double Dl = (double)h->bh[ll] * h->bw[ll], Cin = h->ch[ll], Co = h->ch[ll + 1];
    const double folded = (double)M * Dl * F * Cin * Co + pairs * (F * Cin * Co + (double)O * O * Co);
    if (folded < inside_out_cost(pairs, (int)Dl, h->ch[ll], h->ch[ll + 1], Oe, trace)) inside[ll] = 0;
  }
  fold = fold && !inside[ll];
  // columns of J in this call: per layer its weight block (unless contracted inside-out or
  // folded), then its bias
  std::vector<long long> jw(nc, 0), jb(nc, 0);
  long long Kcall = 0;
  auto plan_columns = [&]() {
    Kcall = 0;
    for (int l = 0; l < nc; ++l) {
      const ntk_layer_desc& L = h->layers[l];
      if (L.kind == NTK_AVGPOOL2) continue;
      if (!inside[l] && !(fold && l == ll)) {
        jw[l] = Kcall;
        Kcall += weight_cols(L, h->ch[l]);
      }
      if (L.has_bias) {
        jb[l] = Kcall;
        Kcall += L.out;
      }
    }
  };
  plan_columns();
  if (fold && Kcall == 0) {
    fold = false;
    plan_columns();
  }
  hipError_t e;
  // 1. forward pass keeping every spatial layer's input, then global average pooling
  const float* h0 = nullptr;
  int rc0 = cnn_forward(h, params, X1, n1, X2, n2, sym, &h0);
  if (rc0 != NTK_OK) return rc0;
  auto hptr = [&](int l) -> const float* { return l == 0 ? h0 : F(h->off_ch[l]); };
  const int C = h->ch[nc];
  // readout summand: (g1 . g2) delta_{o1 o2} ([n1, n2], or [n] on the batch diagonal)
  const float* g2p = sym ? F(h->off_g) : F(h->off_g) + (size_t)n1 * C;
  if (diag) {
    RowdotBatch rb{};
    rb.count = 1;
    rb.a[0] = F(h->off_g);
    rb.b[0] = g2p;
    rb.out[0] = F(h->off_gram_r);
    rb.K[0] = C;
    rb.beta[0] = 0.f;
    prof_begin(P, s, KC_GRAM);
    e = launch_rowdot(s, rb, n1);
    prof_end(P, s, KC_GRAM);
  } else {
    GramBatch gb{};
    gb.count = 1;
    gb.h1[0] = F(h->off_g);
    gb.h2[0] = g2p;
    gb.out[0] = F(h->off_gram_r);
    gb.K[0] = C;
    gb.beta[0] = 0.f;
    prof_begin(P, s, KC_GRAM);
    e = launch_gram(s, gb, n1, n2, h->num_cu);
    prof_end(P, s, KC_GRAM);
  }
  if (e != hipSuccess) return hip_fail(h, e, "gram");
  // 2. cotangents of every spatial layer's output for all O outputs, and per layer its
  //    weight-space cotangent columns of J (or its inside-out summand)
  {
    // the flipped 3x3 kernels and transposed pointwise ones of the backward, in one launch
    FlipBatch fb{};
    for (int l = 1; l < nc; ++l) {
      const int kind = h->layers[l].kind;
      if (kind != NTK_CONV3X3_SAME && kind != NTK_CONV1X1) continue;
      fb.K[fb.count] = params[h->wslot[l]];
      fb.Kt[fb.count] = F(h->off_Kt[l]);
      fb.Cout[fb.count] = h->ch[l + 1];
      fb.Cin[fb.count] = h->ch[l];
      fb.taps[fb.count] = kind == NTK_CONV3X3_SAME ? 9 : 1;
      ++fb.count;
    }
    prof_begin(P, s, KC_TRANSPOSE);
    e = launch_conv_flip_batch(s, fb);
    prof_end(P, s, KC_TRANSPOSE);
    if (e != hipSuccess) return hip_fail(h, e, "kernel flips / transposes");
  }
  float* Gcur = F(h->off_Gping);
  float* Gnext = F(h->off_Gpong);
  prof_begin(P, s, KC_CONV_SEED);
  const float* Wd = params[h->rslot] + (logit ? (size_t)h->opt_logit * C : 0);
  const float* dlast = h->wslot[nc - 1] >= 0 ? F(h->off_cdphi[nc - 1]) : nullptr;
  e = launch_conv_seed(s, Wd, dlast, M, Oe, h->bh[nc] * h->bw[nc], C, Gcur);
  prof_end(P, s, KC_CONV_SEED);
  if (e != hipSuccess) return hip_fail(h, e, "conv seed");
  // weight-space product of layer l's 3x3 (pw: pointwise) convolution: inputs with Cin % 4 != 0
  // padded to the direct-to-LDS form when possible
  auto wgrad = [&](int l, const float* G, int Orows, float* Jout, long long ldJ, long long off, bool pw) {
    const int Hl = h->bh[l], Wl = h->bw[l], cin = h->ch[l], cout = h->ch[l + 1];
    float* xp = h->off_xpad ? F(h->off_xpad) : nullptr;
    if (xp && conv_wgrad_pad_ok(M, Orows, Hl, Wl, cout, cin, G, xp))
      return launch_conv_wgrad_padded(s, G, hptr(l), xp, M, Orows, Hl, Wl, cout, cin, Jout, ldJ, off, pw);
    return pw ? launch_pw_wgrad(s, G, hptr(l), M, Orows, Hl, Wl, cout, cin, Jout, ldJ, off)
              : launch_conv_wgrad(s, G, hptr(l), M, Orows, Hl, Wl, cout, cin, Jout, ldJ, off);
  };
  float* J = F(h->off_J);
  // the folded layer's A: in J past this call's columns (J holds that layer's O C F Cin columns
  // per row), at a 16-byte boundary
  float* fold_A = J + (((size_t)M * Oe * Kcall + 3) & ~(size_t)3);
  bool theta_written = false;
  const int n2_off = sym ? 0 : n1;
  for (int l = nc - 1; l >= 0; --l) {
    const ntk_layer_desc& L = h->layers[l];
    const int Hl = h->bh[l], Wl = h->bw[l], cin = h->ch[l], cout = h->ch[l + 1];
    const float* w = h->wslot[l] >= 0 ? params[h->wslot[l]] : nullptr;
    // Gcur: the cotangent of layer l's pre-activation (of its output for a pool), [M*Oe, ., ., cout]
    if (fold && l == ll) {
      // A [M, C, F Cin] from act'(z) in place of the O cotangents (the "fold" above), in J past
      // the columns of this call
      const float* dz = F(h->off_cdphi[ll]);
      prof_begin(P, s, KC_CONV_WGRAD);
      e = L.kind == NTK_CONV3X3_SAME ? wgrad(l, dz, 1, fold_A, 9LL * cin * cout, 0, false)
                                     : wgrad(l, dz, 1, fold_A, (long long)cin * cout, 0, true);
      prof_end(P, s, KC_CONV_WGRAD);
      if (e != hipSuccess) return hip_fail(h, e, "last convolution's channel cotangents");
      if (L.has_bias) {
        prof_begin(P, s, KC_STRUCT_WGRAD);
        e = launch_pix_wgrad(s, Gcur, nullptr, M, Oe, Hl, Wl, cout, 0, 1, J, Kcall, 0, jb[l], nullptr, 0);
        prof_end(P, s, KC_STRUCT_WGRAD);
        if (e != hipSuccess) return hip_fail(h, e, "conv bias cotangent");
      }
    } else if (L.kind == NTK_CONV3X3_SAME) {
      if (inside[l]) {
        prof_begin(P, s, KC_CONV_PAIRSUM);
        e = launch_conv_pairsum(s, hptr(l), Gcur, F(h->off_gt), n1, n2, n2_off, Oe, Hl, Wl, cin, cout, 9,
                                F(h->off_gram_r), theta_written ? 1 : 0, trace ? 1 : 0, diag ? 1 : 0, theta);
        prof_end(P, s, KC_CONV_PAIRSUM);
        if (e != hipSuccess) return hip_fail(h, e, "conv inside-out pair sum");
        theta_written = true;
      } else {
        prof_begin(P, s, KC_CONV_WGRAD);
        e = wgrad(l, Gcur, Oe, J, Kcall, jw[l], false);
        prof_end(P, s, KC_CONV_WGRAD);
        if (e != hipSuccess) return hip_fail(h, e, "conv weight-space cotangent");
      }
      if (L.has_bias) {
        prof_begin(P, s, KC_STRUCT_WGRAD);
        e = launch_pix_wgrad(s, Gcur, nullptr, M, Oe, Hl, Wl, cout, 0, 1, J, Kcall, 0, jb[l], nullptr, 0);
        prof_end(P, s, KC_STRUCT_WGRAD);
        if (e != hipSuccess) return hip_fail(h, e, "conv bias cotangent");
      }
    } else if (L.kind == NTK_CONV1X1) {
      if (inside[l]) {
        prof_begin(P, s, KC_CONV_PAIRSUM);
        e = launch_conv_pairsum(s, hptr(l), Gcur, F(h->off_gt), n1, n2, n2_off, Oe, Hl, Wl, cin, cout, 1,
                                F(h->off_gram_r), theta_written ? 1 : 0, trace ? 1 : 0, diag ? 1 : 0, theta);
        prof_end(P, s, KC_CONV_PAIRSUM);
        theta_written = true;
      } else {
        prof_begin(P, s, KC_CONV_WGRAD);
        e = wgrad(l, Gcur, Oe, J, Kcall, jw[l], true);
        prof_end(P, s, KC_CONV_WGRAD);
      }
      if (e == hipSuccess && L.has_bias) {
        prof_begin(P, s, KC_STRUCT_WGRAD);
        e = launch_pix_wgrad(s, Gcur, nullptr, M, Oe, Hl, Wl, cout, 0, 1, J, Kcall, 0, jb[l], nullptr, 0);
        prof_end(P, s, KC_STRUCT_WGRAD);
      }
      if (e != hipSuccess) return hip_fail(h, e, "pointwise weight-space cotangent");
    } else if (L.kind != NTK_AVGPOOL2) {
      prof_begin(P, s, KC_STRUCT_WGRAD);
      e = launch_pix_wgrad(s, Gcur, hptr(l), M, Oe, Hl, Wl, cout, L.kind == NTK_DWCONV3X3_SAME ? 9 : 1,
                           L.has_bias, J, Kcall, jw[l], jb[l], F(h->off_part), h->part_capacity);
      prof_end(P, s, KC_STRUCT_WGRAD);
      if (e != hipSuccess) return hip_fail(h, e, "depthwise / scale weight-space cotangent");
    }
    if (l >= 1) {
      // to the cotangent of layer l-1's pre-activation (its output, when it has no activation)
      const float* dprev = h->wslot[l - 1] >= 0 ? F(h->off_cdphi[l - 1]) : nullptr;
      if (L.kind == NTK_CONV3X3_SAME) {
        prof_begin(P, s, KC_CONV_BWD);
        e = launch_conv_bwd(s, Gcur, M, Oe, Hl, Wl, cout, F(h->off_Kt[l]), cin, dprev, Gnext);
        prof_end(P, s, KC_CONV_BWD);
      } else if (L.kind == NTK_CONV1X1) {
        prof_begin(P, s, KC_CONV_BWD);
        int rows;
        e = to_int((long long)M * Oe * Hl * Wl, rows)
                ? launch_pw_bwd(s, Gcur, F(h->off_Kt[l]), dprev, rows, cin, cout, Oe, Hl * Wl, Gnext)
                : hipErrorInvalidValue;
        prof_end(P, s, KC_CONV_BWD);
      } else {
        prof_begin(P, s, KC_STRUCT_BWD);
        if (L.kind == NTK_DWCONV3X3_SAME)
          e = launch_dw_bwd(s, Gcur, M, Oe, Hl, Wl, cout, w, dprev, Gnext);
        else if (L.kind == NTK_SCALE)
          e = launch_scale_bwd(s, Gcur, M, Oe, Hl * Wl, cout, w, dprev, Gnext);
        else
          e = launch_pool_bwd(s, Gcur, M, Oe, Hl, Wl, cin, dprev, Gnext);
        prof_end(P, s, KC_STRUCT_BWD);
      }
      if (e != hipSuccess) return hip_fail(h, e, "backward pass");
      std::swap(Gcur, Gnext);
    }
  }
  // 3. Theta += J1 J2^T over the columns of J (deterministic split over K).  The J rows
  //    of one sample are contiguous, so the traced variant contracts rows (n) of Oe*Kcall
  //    columns; the batch diagonal contracts each sample's rows with its own.
  if (h->opt_method == NTK_METHOD_JACOBIAN) {
    // Jacobian-contraction baseline: the conv layers' explicit J (all of them, outside-in),
    // then the readout layer's explicit block delta_{o o'} g[n, j]
    int rc = ensure_jc_workspace(h);
    if (rc != NTK_OK) return rc;
    const float* J2 = sym ? J : J + (size_t)n1 * Oe * Kcall;
    e = contract_rows(h, J, J2, n1, n2, Oe, trace, diag, sym, Kcall, 0, theta, F(h->off_part),
                      h->part_capacity);
    if (e != hipSuccess) return hip_fail(h, e, "Jacobian contraction");
    bool first = false;
    return jc_dense_layer(h, nullptr, nullptr, 0, F(h->off_g), g2p, C, O, false, n1, n2, Oe,
                          logit ? h->opt_logit : -1, trace, diag, sym, first, theta);
  }
  if (Kcall > 0) {
    const float* J2 = sym ? J : J + (size_t)n1 * Oe * Kcall;
    const float rscale = trace ? (float)O : 1.f;
    if (diag) {
      DiagTerms t{};
      t.count = 1;
      t.A[0] = J;
      t.B[0] = J2;
      t.w[0] = nullptr;
      const bool flat = trace || logit;
      t.K[0] = (flat ? Oe : 1) * Kcall;
      // the readout summand is added once: by the first write of theta
      t.readout = theta_written ? nullptr : F(h->off_gram_r);
      t.readout_scale = rscale;
      prof_begin(P, s, KC_NTK_DIAG);
      e = launch_ntk_diag(s, t, n1, flat ? 0 : O, theta_written ? 1 : 0, theta, F(h->off_part),
                          h->part_capacity);
      prof_end(P, s, KC_NTK_DIAG);
      if (e != hipSuccess) return hip_fail(h, e, "diagonal contraction");
    } else {
      const int Or = trace ? 1 : Oe;                 // rows per sample of the contraction
      const long long Kc = trace ? (long long)O * Kcall : Kcall;
      int R1, R2;
      if (!to_int((long long)n1 * Or, R1) || !to_int((long long)n2 * Or, R2))
        return fail(h, NTK_E_UNSUPPORTED, "contraction rows exceed 2^31");
      int chunk = 0;
      const int splits = splitk_plan(R1, R2, Kc, sym ? 1 : 0, h->part_capacity, &chunk);
      prof_begin(P, s, KC_NTK_SPLITK);
      e = launch_ntk_splitk(s, J, J2, R1, R2, Kc, Kc, sym ? 1 : 0, chunk, splits, F(h->off_part));
      prof_end(P, s, KC_NTK_SPLITK);
      if (e != hipSuccess) return hip_fail(h, e, "split-K contraction");
      prof_begin(P, s, KC_NTK_REDUCE);
      e = launch_ntk_reduce(s, F(h->off_part), splits, n1, n2, Or, sym ? 1 : 0, nullptr, F(h->off_gram_r),
                            rscale, theta_written ? 1 : 0, theta);
      prof_end(P, s, KC_NTK_REDUCE);
      if (e != hipSuccess) return hip_fail(h, e, "split-K reduction");
    }
  }
  if (fold) {
    // theta += sum_c Wr[o1, c] Wr[o2, c] Mc[c] / D^2, Mc[c] = A1[., c, .] A2[., c, .]^T
    const ntk_layer_desc& L = h->layers[ll];
    const int cin = h->ch[ll], KC = (L.kind == NTK_CONV3X3_SAME ? 9 : 1) * cin;
    const int D = h->bh[nc] * h->bw[nc];
    const float* A2 = sym ? fold_A : fold_A + (size_t)n1 * C * KC;
    // the Grams of every pair [C][n1][n2], or on the batch diagonal [C][n] (n2 = 1 below)
    const int m2 = diag ? 1 : n2;
    prof_begin(P, s, KC_GRAM);
    e = diag ? launch_fold_rowdot(s, fold_A, A2, n1, C, KC, F(h->off_mc))
             : launch_gram_strided(s, fold_A, A2, n1, n2, KC, (long long)C * KC, KC, C, F(h->off_mc));
    if (e == hipSuccess)
      e = trace ? launch_readout_fold_trace(s, params[h->rslot], C, O, F(h->off_mc), n1, m2,
                                            1.f / ((float)D * (float)D), theta)
                : launch_readout_fold(s, params[h->rslot], C, O, F(h->off_mc), n1, m2, 1.f / ((float)D * (float)D),
                                      theta);
    prof_end(P, s, KC_GRAM);
    if (e != hipSuccess) return hip_fail(h, e, "last convolution's summand");
  }
  return NTK_OK;
}


// ------------------------------------------------------------------------------ NTK-vector products
static int ensure_vp_workspace_fcn(ntk_handle* h) {
  if (h->vp_ws) return NTK_OK;
  const int L = h->L;
  size_t off = 0;
  auto take = [&](size_t floats) {
    size_t o = off;
    off = align_up(off + floats * 4);
    return o;
  };
  int dmax = 1;
  for (int d : h->dims) dmax = std::max(dmax, d);
  h->vp_off_tc.assign(L + 1, 0);
  h->vp_off_tcb.assign(L + 1, 0);
  for (int l = 0; l <= L; ++l) {
    h->vp_off_tc[l] = take((size_t)h->dims[l + 1] * h->dims[l]);
    h->vp_off_tcb[l] = take((size_t)h->dims[l + 1]);
  }
  h->vp_off_dT = take((size_t)dmax * h->max_n2);
  h->vp_off_hT = take((size_t)dmax * h->max_n2);
  h->vp_off_t0 = take((size_t)dmax * h->max_n1);
  h->vp_off_t1 = take((size_t)dmax * h->max_n1);
  h->vp_off_ga = take((size_t)dmax * h->max_n1);
  h->vp_off_gb = take((size_t)dmax * h->max_n1);
  h->vp_off_WLt = take((size_t)h->dims[L] * h->out_dim);
  hipError_t e = hipMalloc((void**)&h->vp_ws, off);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    h->vp_ws = nullptr;
    return fail(h, NTK_E_OOM, "NTK-vector product buffers of " + std::to_string(off) + " bytes");
  }
  return NTK_OK;
}

// out [n1, O] = Theta(X1, X2) v for v [n2, O]: theta_c = VJP of batch 2 at v (weight space),
// then the JVP of batch 1 along theta_c (Section 3.3, Eq. "ntk_vp_main").
static int vector_product_fcn(ntk_handle* h, const float* const* params, const float* X1, int n1,
                              const float* X2, int n2, const float* v, float* out) {
  const int L = h->L, O = h->out_dim;
  const bool sym = h->opt_symmetric && X1 == X2 && n1 == n2;
  hipStream_t s = h->stream;
  Profiler* P = &h->prof;
  int rc = ensure_vp_workspace_fcn(h);
  if (rc != NTK_OK) return rc;
  const float* h0 = nullptr;
  rc = fcn_forward(h, params, X1, n1, X2, n2, sym, &h0);
  if (rc != NTK_OK) return rc;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(h->ws + off); };
  auto V = [&](size_t off) { return reinterpret_cast<float*>(h->vp_ws + off); };
  auto hptr = [&](int l) -> const float* { return l == 0 ? h0 : F(h->off_h[l]); };
  const size_t r2 = sym ? 0 : (size_t)n1;   // first row of batch 2 in the stacked arrays
  auto W = [&](int l) { return params[h->param_index[l]]; };
  hipError_t e;
  // ---- VJP of batch 2 at v: cotangents delta_l of every pre-activation z_l (delta_L = v)
  for (int l = 1; l < L; ++l) {
    prof_begin(P, s, KC_TRANSPOSE);
    e = launch_transpose(s, W(l), h->dims[l + 1], h->dims[l], F(h->off_Wt[l]));
    prof_end(P, s, KC_TRANSPOSE);
    if (e != hipSuccess) return hip_fail(h, e, "weight transpose");
  }
  auto delta = [&](int l) -> const float* { return l == L ? v : F(h->off_G[l]); };
  if (L >= 1) {
    prof_begin(P, s, KC_TRANSPOSE);
    e = launch_transpose(s, W(L), O, h->dims[L], V(h->vp_off_WLt));
    prof_end(P, s, KC_TRANSPOSE);
    if (e != hipSuccess) return hip_fail(h, e, "weight transpose");
    for (int l = L; l >= 1; --l) {
      // delta_{l-1} = (delta_l W_l) * act'(z_{l-1}) on the rows of batch 2
      const float* Wt = l == L ? V(h->vp_off_WLt) : F(h->off_Wt[l]);
      prof_begin(P, s, KC_DENSE_BWD);
      e = launch_dense_bwd(s, delta(l), Wt, F(h->off_dphi[l - 1]) + r2 * h->dims[l], n2, h->dims[l],
                           h->dims[l + 1], 1, F(h->off_G[l - 1]));
      prof_end(P, s, KC_DENSE_BWD);
      if (e != hipSuccess) return hip_fail(h, e, "VJP backward");
    }
  }
  // weight-space cotangent: theta_c^l = delta_l^T h2_l, bias part sum_n delta_l[n]
  for (int l = 0; l <= L; ++l) {
    const int dout = h->dims[l + 1], din = h->dims[l];
    prof_begin(P, s, KC_TRANSPOSE);
    e = launch_transpose(s, delta(l), n2, dout, V(h->vp_off_dT));
    if (e == hipSuccess) e = launch_transpose(s, hptr(l) + r2 * din, n2, din, V(h->vp_off_hT));
    prof_end(P, s, KC_TRANSPOSE);
    if (e != hipSuccess) return hip_fail(h, e, "VJP transposes");
    GramBatch gb{};
    gb.count = 1;
    gb.h1[0] = V(h->vp_off_dT);
    gb.h2[0] = V(h->vp_off_hT);
    gb.out[0] = V(h->vp_off_tc[l]);
    gb.K[0] = n2;
    gb.beta[0] = 0.f;
    prof_begin(P, s, KC_GRAM);
    e = launch_gram(s, gb, dout, din, h->num_cu);
    prof_end(P, s, KC_GRAM);
    if (e != hipSuccess) return hip_fail(h, e, "weight-space cotangent");
    if (h->layers[l].has_bias) {
      prof_begin(P, s, KC_VP_ELEMENTWISE);
      e = launch_colsum(s, delta(l), n2, dout, V(h->vp_off_tcb[l]));
      prof_end(P, s, KC_VP_ELEMENTWISE);
      if (e != hipSuccess) return hip_fail(h, e, "bias cotangent");
    }
  }
  // ---- JVP of batch 1 along theta_c: tangent t_l of the layer inputs (t_0 = 0),
  //      z'_l = t_l W_l^T + h1_l theta_c^l^T + b'_l,  t_{l+1} = act'(z_l) * z'_l,  out = z'_L
  float* tcur = V(h->vp_off_t0);
  float* tnext = V(h->vp_off_t1);
  for (int l = 0; l <= L; ++l) {
    const int dout = h->dims[l + 1], din = h->dims[l];
    GramBatch gb{};
    gb.count = l > 0 ? 2 : 1;
    gb.h1[0] = hptr(l);
    gb.h2[0] = V(h->vp_off_tc[l]);
    gb.out[0] = V(h->vp_off_ga);
    gb.K[0] = din;
    gb.beta[0] = 0.f;
    if (l > 0) {
      gb.h1[1] = tcur;
      gb.h2[1] = W(l);
      gb.out[1] = V(h->vp_off_gb);
      gb.K[1] = din;
      gb.beta[1] = 0.f;
    }
    prof_begin(P, s, KC_GRAM);
    e = launch_gram(s, gb, n1, dout, h->num_cu);
    prof_end(P, s, KC_GRAM);
    if (e != hipSuccess) return hip_fail(h, e, "JVP products");
    const float* bias_t = h->layers[l].has_bias ? V(h->vp_off_tcb[l]) : nullptr;
    const bool last = l == L;
    prof_begin(P, s, KC_VP_ELEMENTWISE);
    e = launch_jvp_combine(s, l > 0 ? V(h->vp_off_gb) : nullptr, V(h->vp_off_ga), bias_t,
                           last ? nullptr : F(h->off_dphi[l]), n1, dout, last ? out : tnext);
    prof_end(P, s, KC_VP_ELEMENTWISE);
    if (e != hipSuccess) return hip_fail(h, e, "JVP step");
    std::swap(tcur, tnext);
  }
  return NTK_OK;
}


static int ensure_vp_workspace_cnn(ntk_handle* h) {
  if (h->vp_ws) return NTK_OK;
  const int nc = h->nc, O = h->out_dim, C = h->ch[nc];
  size_t pmax = 1;   // largest image of any layer boundary (pixels x channels)
  for (int b = 0; b <= nc; ++b) pmax = std::max(pmax, (size_t)h->bh[b] * h->bw[b] * h->ch[b]);
  size_t off = 0;
  auto take = [&](size_t floats) {
    size_t o = off;
    off = align_up(off + floats * 4);
    return o;
  };
  h->vp_off_tc.assign(1, take((size_t)h->Ktot + (size_t)O * C));   // spatial layers, then the readout
  h->vp_off_dT = take((size_t)O * h->max_n2);
  h->vp_off_hT = take((size_t)C * h->max_n2);
  h->vp_off_WLt = take((size_t)C * O);
  h->vp_off_u = take((size_t)h->max_n2 * C);
  const size_t img = (size_t)h->max_n1 * pmax;
  h->vp_off_t0 = take(img);
  h->vp_off_t1 = take(img);
  h->vp_off_ca = take(img);
  h->vp_off_cb = take(img);
  h->vp_off_cd = take(img);
  h->vp_off_gdot = take((size_t)h->max_n1 * C);
  h->vp_off_ga = take((size_t)h->max_n1 * O);
  h->vp_off_gb = take((size_t)h->max_n1 * O);
  hipError_t e = hipMalloc((void**)&h->vp_ws, off);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    h->vp_ws = nullptr;
    return fail(h, NTK_E_OOM, "NTK-vector product buffers of " + std::to_string(off) + " bytes");
  }
  return NTK_OK;
}

// CNN form of vector_product_fcn: the VJP of batch 2 runs back through the readout, the global
// average pool and the spatial layers, one cotangent row per sample; each layer's weight-space
// cotangent (the same columns the NTK's J holds: a 3x3 convolution's sum_p delta (x) patch, the
// depthwise and scale pixel sums, the bias pixel sums) is formed per sample and summed over the
// samples.  The JVP of batch 1 then pushes that weight-space vector forward: the tangent of a
// parametrised layer's pre-activation is the layer applied to the input tangent plus the layer
// with the tangent weights applied to the input, plus the tangent bias, times act'; a pool
// averages the tangent.
static int vector_product_cnn(ntk_handle* h, const float* const* params, const float* X1, int n1,
                              const float* X2, int n2, const float* v, float* out) {
  const int nc = h->nc, O = h->out_dim, C = h->ch[nc];
  const bool sym = h->opt_symmetric && X1 == X2 && n1 == n2;
  hipStream_t s = h->stream;
  Profiler* P = &h->prof;
  int rc = ensure_vp_workspace_cnn(h);
  if (rc != NTK_OK) return rc;
  const float* h0 = nullptr;
  rc = cnn_forward(h, params, X1, n1, X2, n2, sym, &h0);
  if (rc != NTK_OK) return rc;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(h->ws + off); };
  auto V = [&](size_t off) { return reinterpret_cast<float*>(h->vp_ws + off); };
  auto hptr = [&](int l) -> const float* { return l == 0 ? h0 : F(h->off_ch[l]); };
  auto plane = [&](int b) { return (size_t)h->bh[b] * h->bw[b] * h->ch[b]; };
  const size_t r2 = sym ? 0 : (size_t)n1;   // first row of batch 2 in the stacked arrays
  float* tc = V(h->vp_off_tc[0]);
  float* tc_d = tc + h->Ktot;              // readout part [O, C]
  const float* Wd = params[h->rslot];
  const float* g1 = F(h->off_g);
  const float* g2 = F(h->off_g) + r2 * C;
  const int Dn = h->bh[nc] * h->bw[nc];
  hipError_t e;
  // ---- VJP of batch 2 at v
  prof_begin(P, s, KC_TRANSPOSE);
  e = launch_transpose(s, Wd, O, C, V(h->vp_off_WLt));
  if (e == hipSuccess) e = launch_transpose(s, v, n2, O, V(h->vp_off_dT));
  if (e == hipSuccess) e = launch_transpose(s, g2, n2, C, V(h->vp_off_hT));
  prof_end(P, s, KC_TRANSPOSE);
  if (e != hipSuccess) return hip_fail(h, e, "VJP transposes");
  GramBatch gb{};
  gb.count = 1;
  gb.h1[0] = V(h->vp_off_dT);     // readout weight cotangent v^T g2 [O, C]
  gb.h2[0] = V(h->vp_off_hT);
  gb.out[0] = tc_d;
  gb.K[0] = n2;
  gb.beta[0] = 0.f;
  prof_begin(P, s, KC_GRAM);
  e = launch_gram(s, gb, O, C, h->num_cu);
  prof_end(P, s, KC_GRAM);
  if (e != hipSuccess) return hip_fail(h, e, "readout weight cotangent");
  GramBatch gu{};
  gu.count = 1;                   // u = v W_d [n2, C], the cotangent of the pooled features
  gu.h1[0] = v;
  gu.h2[0] = V(h->vp_off_WLt);
  gu.out[0] = V(h->vp_off_u);
  gu.K[0] = O;
  gu.beta[0] = 0.f;
  prof_begin(P, s, KC_GRAM);
  e = launch_gram(s, gu, n2, C, h->num_cu);
  prof_end(P, s, KC_GRAM);
  if (e != hipSuccess) return hip_fail(h, e, "pooled-feature cotangent");
  float* Gcur = F(h->off_Gping);
  float* Gnext = F(h->off_Gpong);
  const float* dlast = h->wslot[nc - 1] >= 0 ? F(h->off_cdphi[nc - 1]) + r2 * plane(nc) : nullptr;
  prof_begin(P, s, KC_VP_ELEMENTWISE);
  e = launch_gap_adjoint(s, V(h->vp_off_u), dlast, n2, Dn, C, Gcur);
  prof_end(P, s, KC_VP_ELEMENTWISE);
  if (e != hipSuccess) return hip_fail(h, e, "pooling adjoint");
  float* J = F(h->off_J);
  for (int l = nc - 1; l >= 0; --l) {
    const ntk_layer_desc& L = h->layers[l];
    const int Hl = h->bh[l], Wl = h->bw[l], cin = h->ch[l], cout = h->ch[l + 1];
    const float* hl = hptr(l) + r2 * plane(l);
    const float* w = h->wslot[l] >= 0 ? params[h->wslot[l]] : nullptr;
    const long long jw = h->joff[l], jb = jw + weight_cols(L, cin);
    if (L.kind == NTK_CONV3X3_SAME || L.kind == NTK_CONV1X1) {
      prof_begin(P, s, KC_CONV_WGRAD);
      e = L.kind == NTK_CONV3X3_SAME ? launch_conv_wgrad(s, Gcur, hl, n2, 1, Hl, Wl, cout, cin, J, h->Ktot, jw)
                                     : launch_pw_wgrad(s, Gcur, hl, n2, 1, Hl, Wl, cout, cin, J, h->Ktot, jw);
      prof_end(P, s, KC_CONV_WGRAD);
      if (e == hipSuccess && L.has_bias) {
        prof_begin(P, s, KC_STRUCT_WGRAD);
        e = launch_pix_wgrad(s, Gcur, nullptr, n2, 1, Hl, Wl, cout, 0, 1, J, h->Ktot, 0, jb, nullptr, 0);
        prof_end(P, s, KC_STRUCT_WGRAD);
      }
    } else if (L.kind != NTK_AVGPOOL2) {
      prof_begin(P, s, KC_STRUCT_WGRAD);
      e = launch_pix_wgrad(s, Gcur, hl, n2, 1, Hl, Wl, cout, L.kind == NTK_DWCONV3X3_SAME ? 9 : 1, L.has_bias,
                           J, h->Ktot, jw, jb, F(h->off_part), h->part_capacity);
      prof_end(P, s, KC_STRUCT_WGRAD);
    }
    if (e != hipSuccess) return hip_fail(h, e, "VJP weight cotangent");
    if (l >= 1) {
      const float* dprev = h->wslot[l - 1] >= 0 ? F(h->off_cdphi[l - 1]) + r2 * plane(l) : nullptr;
      if (L.kind == NTK_CONV3X3_SAME || L.kind == NTK_CONV1X1) {
        const bool c3 = L.kind == NTK_CONV3X3_SAME;
        prof_begin(P, s, KC_TRANSPOSE);
        e = c3 ? launch_conv_flip(s, w, cout, cin, F(h->off_Kt[l])) : launch_transpose(s, w, cout, cin, F(h->off_Kt[l]));
        prof_end(P, s, KC_TRANSPOSE);
        if (e != hipSuccess) return hip_fail(h, e, "kernel flip / transpose");
        prof_begin(P, s, KC_CONV_BWD);
        e = c3 ? launch_conv_bwd(s, Gcur, n2, 1, Hl, Wl, cout, F(h->off_Kt[l]), cin, dprev, Gnext)
               : launch_pw_bwd(s, Gcur, F(h->off_Kt[l]), dprev, n2 * Hl * Wl, cin, cout, 1, Hl * Wl, Gnext);
        prof_end(P, s, KC_CONV_BWD);
      } else {
        prof_begin(P, s, KC_STRUCT_BWD);
        if (L.kind == NTK_DWCONV3X3_SAME)
          e = launch_dw_bwd(s, Gcur, n2, 1, Hl, Wl, cout, w, dprev, Gnext);
        else if (L.kind == NTK_SCALE)
          e = launch_scale_bwd(s, Gcur, n2, 1, Hl * Wl, cout, w, dprev, Gnext);
        else
          e = launch_pool_bwd(s, Gcur, n2, 1, Hl, Wl, cin, dprev, Gnext);
        prof_end(P, s, KC_STRUCT_BWD);
      }
      if (e != hipSuccess) return hip_fail(h, e, "VJP backward");
      std::swap(Gcur, Gnext);
    }
  }
  prof_begin(P, s, KC_VP_ELEMENTWISE);
  e = launch_colsum(s, J, n2, (int)h->Ktot, tc);   // sum of the per-sample cotangents
  prof_end(P, s, KC_VP_ELEMENTWISE);
  if (e != hipSuccess) return hip_fail(h, e, "weight cotangent sum");
  // ---- JVP of batch 1 along theta_c
  float* tcur = V(h->vp_off_t0);
  float* tnext = V(h->vp_off_t1);
  float* ca = V(h->vp_off_ca);
  float* cb = V(h->vp_off_cb);
  float* cd = V(h->vp_off_cd);   // act' outputs of the activation-free evaluations, unused
  bool tzero = true;             // the tangent of layer l's input is zero (no parameter before it)
  for (int l = 0; l < nc; ++l) {
    const ntk_layer_desc& L = h->layers[l];
    const int Hl = h->bh[l], Wl = h->bw[l], cin = h->ch[l], cout = h->ch[l + 1];
    if (L.kind == NTK_AVGPOOL2) {
      if (tzero) continue;
      prof_begin(P, s, KC_STRUCT_FWD);
      e = launch_pool_fwd(s, tcur, n1, Hl, Wl, cin, tnext);
      prof_end(P, s, KC_STRUCT_FWD);
      if (e != hipSuccess) return hip_fail(h, e, "JVP pool");
      std::swap(tcur, tnext);
      continue;
    }
    const float* w = params[h->wslot[l]];
    const float* tw = tc + h->joff[l];
    const float* tb = L.has_bias ? tc + h->joff[l] + weight_cols(L, cin) : nullptr;
    const float* hl = hptr(l);
    // cb = the layer with the tangent weights applied to the input; ca = the layer applied to
    // the input tangent
    if (L.kind == NTK_CONV3X3_SAME) {
      prof_begin(P, s, KC_CONV_FWD);
      e = launch_conv_fwd(s, hl, n1, Hl, Wl, cin, tw, cout, NTK_ACT_NONE, nullptr, cb, cd);
      if (e == hipSuccess && !tzero)
        e = launch_conv_fwd(s, tcur, n1, Hl, Wl, cin, w, cout, NTK_ACT_NONE, nullptr, ca, cd);
      prof_end(P, s, KC_CONV_FWD);
    } else if (L.kind == NTK_CONV1X1) {
      const int rows = n1 * Hl * Wl;
      prof_begin(P, s, KC_CONV_FWD);
      e = launch_dense_fwd(s, hl, tw, nullptr, rows, cout, cin, NTK_ACT_NONE, cb, cd, nullptr, 0);
      if (e == hipSuccess && !tzero)
        e = launch_dense_fwd(s, tcur, w, nullptr, rows, cout, cin, NTK_ACT_NONE, ca, cd, nullptr, 0);
      prof_end(P, s, KC_CONV_FWD);
    } else {
      prof_begin(P, s, KC_STRUCT_FWD);
      if (L.kind == NTK_DWCONV3X3_SAME) {
        e = launch_dw_fwd(s, hl, n1, Hl, Wl, cin, tw, nullptr, NTK_ACT_NONE, cb, cd);
        if (e == hipSuccess && !tzero) e = launch_dw_fwd(s, tcur, n1, Hl, Wl, cin, w, nullptr, NTK_ACT_NONE, ca, cd);
      } else {
        e = launch_scale_fwd(s, hl, n1, Hl * Wl, cin, tw, nullptr, NTK_ACT_NONE, cb, cd);
        if (e == hipSuccess && !tzero)
          e = launch_scale_fwd(s, tcur, n1, Hl * Wl, cin, w, nullptr, NTK_ACT_NONE, ca, cd);
      }
      prof_end(P, s, KC_STRUCT_FWD);
    }
    if (e != hipSuccess) return hip_fail(h, e, "JVP layer");
    prof_begin(P, s, KC_VP_ELEMENTWISE);
    e = launch_jvp_combine(s, tzero ? nullptr : ca, cb, tb, F(h->off_cdphi[l]), n1 * Hl * Wl, cout, tnext);
    prof_end(P, s, KC_VP_ELEMENTWISE);
    if (e != hipSuccess) return hip_fail(h, e, "JVP step");
    std::swap(tcur, tnext);
    tzero = false;
  }
  prof_begin(P, s, KC_GAP);
  e = launch_gap(s, tcur, n1, Dn, C, V(h->vp_off_gdot));
  prof_end(P, s, KC_GAP);
  if (e != hipSuccess) return hip_fail(h, e, "JVP pooling");
  GramBatch gr{};
  gr.count = 2;                    // out = gdot W_d^T + g1 theta_c^d^T
  gr.h1[0] = V(h->vp_off_gdot);
  gr.h2[0] = Wd;
  gr.out[0] = V(h->vp_off_ga);
  gr.K[0] = C;
  gr.beta[0] = 0.f;
  gr.h1[1] = g1;
  gr.h2[1] = tc_d;
  gr.out[1] = V(h->vp_off_gb);
  gr.K[1] = C;
  gr.beta[1] = 0.f;
  prof_begin(P, s, KC_GRAM);
  e = launch_gram(s, gr, n1, O, h->num_cu);
  prof_end(P, s, KC_GRAM);
  if (e != hipSuccess) return hip_fail(h, e, "JVP readout");
  prof_begin(P, s, KC_VP_ELEMENTWISE);
  e = launch_jvp_combine(s, V(h->vp_off_ga), V(h->vp_off_gb), nullptr, nullptr, n1, O, out);
  prof_end(P, s, KC_VP_ELEMENTWISE);
  if (e != hipSuccess) return hip_fail(h, e, "JVP output");
  return NTK_OK;
}

static int compute_eager(ntk_handle* h, const float* const* params, const float* X1, int n1, const float* X2,
                         int n2, float* theta) {
  if (h->cnn) return compute_cnn(h, params, X1, n1, X2, n2, theta);
  return compute_fcn(h, params, X1, n1, X2, n2, theta);
}

static int param_tensor_count(const ntk_handle* h) {
  if (h->cnn) return h->rslot + 1;
  int n = 0;
  for (const auto& L : h->layers) n += 1 + (L.has_bias ? 1 : 0);
  return n;
}

// NTK_OPT_GRAPH: replay the recorded graph when every argument and option matches, else record.
static int compute_graph(ntk_handle* h, const float* const* params, const float* X1, int n1, const float* X2,
                         int n2, float* theta) {
  std::vector<uintptr_t> key;
  const int np = param_tensor_count(h);
  for (int i = 0; i < np; ++i) key.push_back(reinterpret_cast<uintptr_t>(params[i]));
  for (uintptr_t v : {reinterpret_cast<uintptr_t>(X1), reinterpret_cast<uintptr_t>(X2),
                      reinterpret_cast<uintptr_t>(theta), reinterpret_cast<uintptr_t>(h->stream)})
    key.push_back(v);
  for (int v : {n1, n2, h->opt_symmetric, h->opt_conv_order, h->opt_output, h->opt_logit, h->opt_batch,
                h->opt_method})
    key.push_back((uintptr_t)(unsigned)v);
  hipError_t e;
  if (!h->gstream) {
    if ((e = hipStreamCreateWithFlags(&h->gstream, hipStreamNonBlocking)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&h->ev_gin, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&h->ev_gout, hipEventDisableTiming)) != hipSuccess)
      return hip_fail(h, e, "graph stream");
  }
  const hipStream_t user = h->stream;
  // the graph's work starts after everything enqueued on the caller's stream so far
  if ((e = hipEventRecord(h->ev_gin, user)) != hipSuccess ||
      (e = hipStreamWaitEvent(h->gstream, h->ev_gin, 0)) != hipSuccess)
    return hip_fail(h, e, "graph stream fork");
  if (!(h->graph_exec && key == h->graph_key)) {
    if (h->graph_exec) (void)hipGraphExecDestroy(h->graph_exec);
    h->graph_exec = nullptr;
    h->graph_key.clear();
    if (h->opt_method == NTK_METHOD_JACOBIAN) {   // no allocation while recording
      int rc = ensure_jc_workspace(h);
      if (rc != NTK_OK) return rc;
    }
    // relaxed: the launchers set kernel attributes (LDS size), which is not a stream operation
    if ((e = hipStreamBeginCapture(h->gstream, hipStreamCaptureModeRelaxed)) != hipSuccess)
      return hip_fail(h, e, "graph capture");
    h->stream = h->gstream;
    const int rc = compute_eager(h, params, X1, n1, X2, n2, theta);
    h->stream = user;
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(h->gstream, &g);
    if (rc != NTK_OK) {
      if (g) (void)hipGraphDestroy(g);
      return rc;
    }
    if (e != hipSuccess) return hip_fail(h, e, "graph capture");
    e = hipGraphInstantiate(&h->graph_exec, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) {
      h->graph_exec = nullptr;
      return hip_fail(h, e, "graph instantiation");
    }
    h->graph_key = key;
  }
  if ((e = hipGraphLaunch(h->graph_exec, h->gstream)) != hipSuccess) return hip_fail(h, e, "graph launch");
  // and the caller's later work waits for the graph
  if ((e = hipEventRecord(h->ev_gout, h->gstream)) != hipSuccess ||
      (e = hipStreamWaitEvent(user, h->ev_gout, 0)) != hipSuccess)
    return hip_fail(h, e, "graph stream join");
  return NTK_OK;
}

extern "C" int ntk_compute(ntk_handle* h, const float* const* params, const float* X1, int n1,
                           const float* X2, int n2, float* theta) {
  if (!h) return fail(nullptr, NTK_E_ARG, "handle is NULL");
  if (!params || !X1 || !X2 || !theta) return fail(h, NTK_E_ARG, "null pointer argument");
  if (n1 <= 0 || n2 <= 0) return fail(h, NTK_E_ARG, "n1 and n2 must be positive");
  if (n1 > h->max_n1 || n2 > h->max_n2)
    return fail(h, NTK_E_ARG, "n1/n2 exceed the max_n1/max_n2 given to ntk_init");
  if (h->opt_output == NTK_OUTPUT_LOGIT && h->opt_logit >= h->out_dim)
    return fail(h, NTK_E_ARG, "NTK_OPT_LOGIT must be below the number of outputs");
  if (h->opt_batch == NTK_BATCH_DIAGONAL && n1 != n2)
    return fail(h, NTK_E_ARG, "NTK_BATCH_DIAGONAL needs n1 == n2");
  const int np = param_tensor_count(h);
  for (int i = 0; i < np; ++i)
    if (!params[i]) return fail(h, NTK_E_ARG, "null parameter pointer");
  h->err.clear();
  if (h->opt_graph && !h->prof.enabled) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(h->stream, &st) == hipSuccess && st == hipStreamCaptureStatusNone)
      return compute_graph(h, params, X1, n1, X2, n2, theta);
  }
  return compute_eager(h, params, X1, n1, X2, n2, theta);
}

// ------------------------------------------------------------------------------ no-allocation entry
// The workspace of ntk_compute_static: one array per device, resident until the process ends.
// In host code `scratch` names a host-side stand-in, not the device array, so it is never passed
// to a kernel or a copy; the device address comes from hipGetSymbolAddress, once per device, on
// the first call made with that device current.
static __device__ __align__(256) char scratch[NTK_STATIC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static char* g_scratch_ptr[kMaxDevices] = {};

static int static_scratch(char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(nullptr, e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(nullptr, NTK_E_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(nullptr, e, "hipGetSymbolAddress of the static scratch");
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return NTK_OK;
}

extern "C" int ntk_compute_static(const ntk_model_desc* model, const float* const* params, const float* X1,
                                  int n1, const float* X2, int n2, float* theta, void* hip_stream) {
  if (!params || !X1 || !X2 || !theta) return fail(nullptr, NTK_E_ARG, "null pointer argument");
  if (n1 <= 0 || n2 <= 0) return fail(nullptr, NTK_E_ARG, "n1 and n2 must be positive");
  // a handle on the stack: host bookkeeping only, no streams, events or device memory
  ntk_handle h;
  int rc = validate(model, &h);
  if (rc != NTK_OK) return rc;
  h.layers.assign(model->layers, model->layers + model->n_layers);
  h.in_h = model->in_h;
  h.in_w = model->in_w;
  h.in_c = model->in_c;
  h.out_dim = model->out_dim;
  rc = check_index_range(h, n1, n2);
  if (rc != NTK_OK) return rc;
  h.max_n1 = n1;
  h.max_n2 = n2;
  h.lean = true;
  if (h.cnn)
    plan_cnn(&h);
  else
    plan_fcn(&h);
  if (h.ws_bytes > (size_t)NTK_STATIC_SCRATCH_BYTES)
    return fail(nullptr, NTK_E_UNSUPPORTED,
                "this model and these batch sizes need " + std::to_string(h.ws_bytes) +
                    " bytes of workspace; the static scratch holds " + std::to_string(NTK_STATIC_SCRATCH_BYTES) +
                    " (use ntk_init and ntk_compute)");
  const int np = param_tensor_count(&h);
  for (int i = 0; i < np; ++i)
    if (!params[i]) return fail(nullptr, NTK_E_ARG, "null parameter pointer");
  rc = static_scratch(&h.ws);
  if (rc != NTK_OK) return rc;
  h.stream = (hipStream_t)hip_stream;
  rc = compute_eager(&h, params, X1, n1, X2, n2, theta);
  h.ws = nullptr;   // the scratch is never released
  if (rc != NTK_OK) g_init_error = h.err;
  return rc;
}

extern "C" int ntk_vector_product(ntk_handle* h, const float* const* params, const float* X1, int n1,
                                  const float* X2, int n2, const float* v, float* out) {
  if (!h) return fail(nullptr, NTK_E_ARG, "handle is NULL");
  if (!params || !X1 || !X2 || !v || !out) return fail(h, NTK_E_ARG, "null pointer argument");
  if (n1 <= 0 || n2 <= 0) return fail(h, NTK_E_ARG, "n1 and n2 must be positive");
  if (n1 > h->max_n1 || n2 > h->max_n2)
    return fail(h, NTK_E_ARG, "n1/n2 exceed the max_n1/max_n2 given to ntk_init");
  h->err.clear();
  if (h->cnn) return vector_product_cnn(h, params, X1, n1, X2, n2, v, out);
  return vector_product_fcn(h, params, X1, n1, X2, n2, v, out);
}

extern "C" int ntk_free(ntk_handle* h) {
  if (!h) return NTK_OK;
  (void)hipStreamSynchronize(h->stream);
  if (h->graph_exec) (void)hipGraphExecDestroy(h->graph_exec);
  if (h->gstream) (void)hipStreamSynchronize(h->gstream);
  if (h->ev_gin) (void)hipEventDestroy(h->ev_gin);
  if (h->ev_gout) (void)hipEventDestroy(h->ev_gout);
  if (h->gstream) (void)hipStreamDestroy(h->gstream);
  if (h->ws) (void)hipFree(h->ws);
  destroy_sync_objects(h);
  if (h->jc_ws) (void)hipFree(h->jc_ws);
  if (h->vp_ws) (void)hipFree(h->vp_ws);
  delete h;
  return NTK_OK;
}

extern "C" const char* ntk_last_error(const ntk_handle* h) {
  return h ? h->err.c_str() : g_init_error.c_str();
}

extern "C" int ntk_set_option(ntk_handle* h, int option, int value) {
  if (!h) return fail(nullptr, NTK_E_ARG, "handle is NULL");
  if (option == NTK_OPT_SYMMETRIC) {
    if (value != 0 && value != 1) return fail(h, NTK_E_ARG, "NTK_OPT_SYMMETRIC takes 0 or 1");
    h->opt_symmetric = value;
    return NTK_OK;
  }
  if (option == NTK_OPT_CONV_ORDER) {
    if (value < NTK_CONV_ORDER_AUTO || value > NTK_CONV_ORDER_INSIDE_OUT)
      return fail(h, NTK_E_ARG, "NTK_OPT_CONV_ORDER takes 0, 1 or 2");
    h->opt_conv_order = value;
    return NTK_OK;
  }
  if (option == NTK_OPT_OUTPUT) {
    if (value != NTK_OUTPUT_FULL && value != NTK_OUTPUT_TRACE && value != NTK_OUTPUT_LOGIT)
      return fail(h, NTK_E_ARG, "NTK_OPT_OUTPUT takes NTK_OUTPUT_FULL, _TRACE or _LOGIT");
    h->opt_output = value;
    return NTK_OK;
  }
  if (option == NTK_OPT_LOGIT) {
    if (value < 0 || value >= h->out_dim) return fail(h, NTK_E_ARG, "NTK_OPT_LOGIT must be in [0, O)");
    h->opt_logit = value;
    return NTK_OK;
  }
  if (option == NTK_OPT_METHOD) {
    if (value != NTK_METHOD_STRUCTURED && value != NTK_METHOD_JACOBIAN)
      return fail(h, NTK_E_ARG, "NTK_OPT_METHOD takes NTK_METHOD_STRUCTURED or NTK_METHOD_JACOBIAN");
    h->opt_method = value;
    return NTK_OK;
  }
  if (option == NTK_OPT_GRAPH) {
    if (value != 0 && value != 1) return fail(h, NTK_E_ARG, "NTK_OPT_GRAPH takes 0 or 1");
    h->opt_graph = value;
    if (!value && h->graph_exec) {
      (void)hipGraphExecDestroy(h->graph_exec);
      h->graph_exec = nullptr;
      h->graph_key.clear();
    }
    return NTK_OK;
  }
  if (option == NTK_OPT_BATCH) {
    if (value != NTK_BATCH_FULL && value != NTK_BATCH_DIAGONAL)
      return fail(h, NTK_E_ARG, "NTK_OPT_BATCH takes NTK_BATCH_FULL or NTK_BATCH_DIAGONAL");
    h->opt_batch = value;
    return NTK_OK;
  }
  return fail(h, NTK_E_ARG, "unknown option");
}

extern "C" int ntk_set_stream(ntk_handle* h, void* hip_stream) {
  if (!h) return fail(nullptr, NTK_E_ARG, "handle is NULL");
  h->stream = (hipStream_t)hip_stream;
  return NTK_OK;
}

extern "C" long long ntk_workspace_bytes(const ntk_handle* h) { return h ? (long long)h->ws_bytes : 0; }

extern "C" int ntk_profile_enable(ntk_handle* h, int enable) {
  if (!h) return fail(nullptr, NTK_E_ARG, "handle is NULL");
  h->prof.enabled = enable != 0;
  return NTK_OK;
}

extern "C" int ntk_profile_read(ntk_handle* h, const char** names, double* total_ms, long long* launches,
                                int max) {
  if (!h) return fail(nullptr, NTK_E_ARG, "handle is NULL");
  if (max < 0 || (max > 0 && (!names || !total_ms || !launches))) return fail(h, NTK_E_ARG, "bad output arrays");
  hipError_t e = hipStreamSynchronize(h->stream);
  if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
  Profiler& p = h->prof;
  for (auto& q : p.pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, q.a, q.b) == hipSuccess) {
      p.total_ms[q.cls] += ms;
      p.launches[q.cls] += 1;
    }
    p.pool.push_back(q.a);
    p.pool.push_back(q.b);
  }
  p.pending.clear();
  int n = 0;
  for (int c = 0; c < KC_COUNT && n < max; ++c) {
    if (p.launches[c] == 0) continue;
    names[n] = kernel_class_name(c);
    total_ms[n] = p.total_ms[c];
    launches[n] = p.launches[c];
    ++n;
  }
  for (int c = 0; c < KC_COUNT; ++c) {
    p.total_ms[c] = 0;
    p.launches[c] = 0;
  }
  return n;
}
