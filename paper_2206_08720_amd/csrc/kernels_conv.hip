// kernels_conv.hip -- convolutional path of the structured-derivatives NTK on gfx950.
//
// A 3x3 SAME, stride-1 convolution z[p, c] = sum_k patch[p, k] K[c, k] has a
// Jacobian dz/dK that is constant-block diagonal along the output channel (the
// appendix "Constant-block Diagonal" structure, C = W for a convolution), so the
// smallest sub-array to keep is the patch matrix of the layer input (appendix
// "CNN NTK Complexity": D x F*Cin per sample, formed here implicitly inside the
// GEMM loaders).  The kernels compute
//   * the forward pass keeping every layer input and act'(z) (fp64 accumulation, as
//     for dense layers, so ReLU decisions are a function of the fp32-stored input)
//   * global average pooling (the input block-tiled structure of a mean)
//   * the cotangent of the last conv pre-activation, W_d[o, c] / D * act'(z)
//   * the transposed convolution pulling the (N1+N2)*O cotangent images back one
//     layer (a SAME convolution with the spatially flipped, channel-transposed kernel)
//   * the outside-in weight-sharing contraction: per sample and layer the weight-space
//     cotangent J[(n,o),(c,k)] = sum_p G[n,o,p,c] patch[n,p,k]
//   * J1 J2^T with a deterministic split over K, then a reduction adding the readout
//     summand (g1.g2) delta_{o1 o2} and writing theta[n1][n2][o1][o2].
#include <type_traits>

#include "gemm_core.hpp"
#include "launch_conv.hpp"

namespace ntk {

using CfgConvF64 = TileCfg<64, 64, 32, 32, 32>;    // forward, fp64 MFMA
using CfgConv = TileCfg<128, 64, 32, 32, 32>;      // backward / wgrad, fp32 MFMA: 8 waves
// direct-to-LDS backward and weight-space cotangent kernels: tiles and LDS stages.  The
// backward takes 256-row tiles with a 32x64 block per wave (two independent accumulators per
// wave) and two stages (80 KB: two workgroups per CU); the weight-space product keeps 128x64
// tiles and two stages (48 KB: three workgroups per CU).  Both measured best among 128/256-row
// tiles, 4/8 waves and 2/3 stages at the CNN workload.
using CfgConvBwd = TileCfg<256, 64, 32, 32, 64>;
using CfgConvWg = CfgConv;
using CfgConvWgSmall = TileCfg<64, 64, 32, 32, 32>;   // one-output rows (O C <= 64): 4 waves
constexpr int kConvBwdStages = 2, kConvWgStages = 2;
// Small images (few output rows): below kConvFewTiles tiles of the shapes above, the backward
// takes 128x64 tiles (8 waves of 32x32) and the fp64 forward 32x32 tiles (4 waves of 16x16), so
// that the launch still spreads over the compute units.
constexpr int kConvFewTiles = 512;
using CfgConvF64Small = TileCfg<32, 32, 32, 16, 16>;
using CfgSplitK = TileCfg<128, 128, 32, 64, 64>;   // J1 J2^T partial products
using CfgSplitKDma = TileCfg<128, 128, 32, 32, 64>;  // the same, direct-to-LDS: 8 waves of 32x64

static inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }
static inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <class Cfg, class LA, class LB>
static hipError_t set_smem(const void* fn) {
  constexpr int bytes = gemm_smem_bytes<Cfg, LA, LB>();
  if (bytes > 65536)
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  return hipSuccess;
}

// ------------------------------------------------------------------------------ loaders
// All loaders read from clamped in-range addresses and report per-element validity (bit j
// of `valid`); the zero fill happens at the LDS store (see TileIO).
//
// Patch matrix of an NHWC batch as a K-inner operand: row = img*D + p, p = y*W + x,
// k = (kh*3 + kw)*C + ci; the tap (kh, kw) reads pixel (y + kh - 1, x + kw - 1), zero
// outside the image.  VEC: C % 4 == 0 and x 16-byte aligned (4 k share one tap).
template <bool VEC>
struct LoadPatchesKInnerT {
  static constexpr bool K_INNER = true;
  static constexpr bool UNIFORM_VALID = VEC;   // VEC: the 4 elements are valid together
  const float* x;
  int rows, H, W, C, K;  // K = 9*C
  FastDiv fD, fW, fC;
  __device__ __forceinline__ float tap(int img, int y, int xx, int k, bool& ok) const {
    const int kc = min(k, K - 1);
    const int t = (int)fC.div(kc), ci = kc - t * C;
    const int kh = (t * 11) >> 5, kw = t - 3 * kh;  // t / 3 for t < 9
    const int yy = y + kh - 1, xq = xx + kw - 1;
    ok = k < K && yy >= 0 && yy < H && xq >= 0 && xq < W;
    const int yc = min(max(yy, 0), H - 1), xc = min(max(xq, 0), W - 1);
    return x[(((long long)img * H + yc) * W + xc) * C + ci];
  }
  // the row's pixel, computed once per tile: element offset of (img, y, x) (clamped row), y, x
  struct RowState {
    long long base;
    int y, x, ok;
  };
  __device__ __forceinline__ RowState row_state(int row) const {
    const int rc = min(row, rows - 1);
    const int img = (int)fD.div(rc), p = rc - img * (int)fD.d;
    const int y = (int)fW.div(p), xx = p - y * W;
    return {(((long long)img * H + y) * W + xx) * C, y, xx, row < rows ? 1 : 0};
  }
  // element (row, k): tap (kh, kw) = k / C reads the pixel (y + kh - 1, x + kw - 1); outside the
  // image the row's own pixel is read and masked
  __device__ __forceinline__ f32x4 load4s(const RowState& s, int k, uint32_t& valid) const {
    if (VEC) {
      const int kc = min(k, K - 4);
      const int t = (int)fC.div(kc), ci = kc - t * C;
      const int kh = (t * 11) >> 5, kw = t - 3 * kh;
      const int yy = s.y + kh - 1, xq = s.x + kw - 1;
      const bool ok = s.ok & (k < K) & ((unsigned)yy < (unsigned)H) & ((unsigned)xq < (unsigned)W);
      const int off = ok ? ((kh - 1) * W + (kw - 1)) * C + ci : ci;
      valid = ok ? 0xFu : 0u;
      return *reinterpret_cast<const f32x4*>(x + s.base + off);
    } else {
      f32x4 v;
      valid = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kc = min(k + j, K - 1);
        const int t = (int)fC.div(kc), ci = kc - t * C;
        const int kh = (t * 11) >> 5, kw = t - 3 * kh;
        const int yy = s.y + kh - 1, xq = s.x + kw - 1;
        const bool ok = s.ok && k + j < K && yy >= 0 && yy < H && xq >= 0 && xq < W;
        const long long off = ok ? (long long)((kh - 1) * W + (kw - 1)) * C : 0;
        v[j] = x[s.base + off + ci];
        valid |= ok ? (1u << j) : 0u;
      }
      return v;
    }
  }
  __device__ __forceinline__ f32x4 load4(int row, int k, uint32_t& valid) const {
    const int rc = min(row, rows - 1);
    const int img = (int)fD.div(rc), p = rc - img * (int)fD.d;
    const int y = (int)fW.div(p), xx = p - y * W;
    if (VEC) {
      const int kc = min(k, K - 4);
      const int t = (int)fC.div(kc), ci = kc - t * C;
      const int kh = (t * 11) >> 5, kw = t - 3 * kh;
      const int yy = y + kh - 1, xq = xx + kw - 1;
      const bool ok = row < rows && k < K && yy >= 0 && yy < H && xq >= 0 && xq < W;
      const int yc = min(max(yy, 0), H - 1), xc = min(max(xq, 0), W - 1);
      valid = ok ? 0xFu : 0u;
      return *reinterpret_cast<const f32x4*>(x + (((long long)img * H + yc) * W + xc) * C + ci);
    } else {
      f32x4 v;
      valid = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bool ok;
        v[j] = tap(img, y, xx, k + j, ok);
        valid |= (ok && row < rows) ? (1u << j) : 0u;
      }
      return v;
    }
  }
};

// G of one sample as a K-outer operand of the weight-space cotangent product:
// row = o*C + c, k = p;  element = G[((s*O + o)*D + p)*C + c]  (base already at sample s).
// VEC: C % 4 == 0 and g 16-byte aligned.
template <bool VEC>
struct LoadCotangentKOuterT {
  static constexpr bool K_INNER = false;
  static constexpr bool UNIFORM_VALID = VEC;
  const float* g;
  int rows, K, C, D;     // rows = O*C, K = D
  FastDiv fC;
  // offset o*D*C + c of the row block (VEC: rows row..row+3 are contiguous), once per tile
  struct RowState {
    long long off;
    int row;
  };
  __device__ __forceinline__ RowState row_state(int row) const {
    const int rc = min(row, VEC ? rows - 4 : rows - 1);
    const int o = (int)fC.div(rc), c = rc - o * C;
    return {(long long)o * D * C + c, row};
  }
  __device__ __forceinline__ f32x4 load4s(const RowState& s, int k, uint32_t& valid) const {
    if (VEC) {
      const int kc = min(k, K - 1);
      valid = (s.row < rows && k < K) ? 0xFu : 0u;
      return *reinterpret_cast<const f32x4*>(g + s.off + (long long)kc * C);
    }
    return load4(s.row, k, valid);
  }
  __device__ __forceinline__ f32x4 load4(int row, int k, uint32_t& valid) const {
    const int kc = min(k, K - 1);
    if (VEC) {
      const int rc = min(row, rows - 4);
      const int o = (int)fC.div(rc), c = rc - o * C;
      valid = (row < rows && k < K) ? 0xFu : 0u;
      return *reinterpret_cast<const f32x4*>(g + ((long long)o * D + kc) * C + c);
    } else {
      f32x4 v;
      valid = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int rc = min(row + j, rows - 1);
        const int o = (int)fC.div(rc), c = rc - o * C;
        v[j] = g[((long long)o * D + kc) * C + c];
        valid |= (row + j < rows && k < K) ? (1u << j) : 0u;
      }
      return v;
    }
  }
};

// Patch matrix of one sample as a K-outer operand: row = k (tap, ci), kdim = p.
// VEC: C % 4 == 0 and x 16-byte aligned.
template <bool VEC>
struct LoadPatchesKOuterT {
  static constexpr bool K_INNER = false;
  static constexpr bool UNIFORM_VALID = VEC;
  const float* x;        // sample base, [H, W, C]
  int rows, K, H, W, C;  // rows = 9*C, K = D
  FastDiv fW, fC;
  // the rows' tap offset (dy, dx) and first channel (VEC: 4 consecutive channels of one
  // tap), once per tile
  struct RowState {
    int dy, dx, dd, ci, row;   // dd = dy * W + dx
  };
  __device__ __forceinline__ RowState row_state(int row) const {
    const int rc = min(row, VEC ? rows - 4 : rows - 1);
    const int t = (int)fC.div(rc), ci = rc - t * C;
    const int kh = (t * 11) >> 5, kw = t - 3 * kh;
    return {kh - 1, kw - 1, (kh - 1) * W + (kw - 1), ci, row};
  }
  __device__ __forceinline__ f32x4 load4s(const RowState& s, int p, uint32_t& valid) const {
    if (VEC) {
      const int pc = min(p, K - 1);
      const int y = (int)fW.div(pc), xx = pc - y * W;
      const int yy = y + s.dy, xq = xx + s.dx;
      const bool ok = (s.row < rows) & (p < K) & ((unsigned)yy < (unsigned)H) & ((unsigned)xq < (unsigned)W);
      valid = ok ? 0xFu : 0u;
      const int q = ok ? pc + s.dd : pc;   // outside the image: the pixel itself, masked
      return *reinterpret_cast<const f32x4*>(x + (long long)q * C + s.ci);
    }
    return load4(s.row, p, valid);
  }
  __device__ __forceinline__ f32x4 load4(int row, int p, uint32_t& valid) const {
    const int pc = min(p, K - 1);
    const int y = (int)fW.div(pc), xx = pc - y * W;
    if (VEC) {
      const int rc = min(row, rows - 4);
      const int t = (int)fC.div(rc), ci = rc - t * C;
      const int kh = (t * 11) >> 5, kw = t - 3 * kh;
      const int yy = y + kh - 1, xq = xx + kw - 1;
      const bool ok = row < rows && p < K && yy >= 0 && yy < H && xq >= 0 && xq < W;
      const int yc = min(max(yy, 0), H - 1), xc = min(max(xq, 0), W - 1);
      valid = ok ? 0xFu : 0u;
      return *reinterpret_cast<const f32x4*>(x + ((long long)yc * W + xc) * C + ci);
    } else {
      f32x4 v;
      valid = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int rc = min(row + j, rows - 1);
        const int t = (int)fC.div(rc), ci = rc - t * C;
        const int kh = (t * 11) >> 5, kw = t - 3 * kh;
        const int yy = y + kh - 1, xq = xx + kw - 1;
        const bool ok = row + j < rows && p < K && yy >= 0 && yy < H && xq >= 0 && xq < W;
        const int yc = min(max(yy, 0), H - 1), xc = min(max(xq, 0), W - 1);
        v[j] = x[((long long)yc * W + xc) * C + ci];
        valid |= ok ? (1u << j) : 0u;
      }
      return v;
    }
  }
};

template <bool VEC>
static LoadPatchesKInnerT<VEC> patches_kinner(const float* x, int images, int H, int W, int C) {
  LoadPatchesKInnerT<VEC> l;
  l.x = x;
  l.rows = images * H * W;
  l.H = H;
  l.W = W;
  l.C = C;
  l.K = 9 * C;
  l.fD = FastDiv((uint32_t)(H * W));
  l.fW = FastDiv((uint32_t)W);
  l.fC = FastDiv((uint32_t)C);
  return l;
}

// Patch matrix of an NHWC batch as a direct-to-LDS operand (see DmaTile): row = img*D + p,
// column k = tap*C + ci with C % 32 == 0, so the 32 columns of a K tile lie inside one tap.
// Every lane loads 16 bytes of one row through a buffer resource over the whole batch (less
// than 2 GiB); a tap that falls outside the image (the zero padding) takes an offset past the
// resource, which reads zeros.  The rows' pixels are computed once per tile (prepare).
constexpr uint32_t kDmaPastEnd = 0x80000000u;   // past every resource: the load reads zeros

template <int ROWS, int WAVES>
struct DmaPatches {
  using Tile = DmaTile<ROWS>;
  const float* __restrict__ x;
  int rows, H, W, C;
  FastDiv fD, fW, fC;
  static constexpr int NI = ROWS / (8 * WAVES);
  template <int WV>
  static constexpr int OPS = ROWS / (8 * WV);
  __amdgpu_buffer_rsrc_t rsrc;
  // per issued row: the byte offset of its pixel's 16-byte chunk (channel block 0) through a
  // resource that starts W + 1 pixels before the batch, so that every tap's shift is a
  // non-negative uniform offset (the scalar offset of the load), and a 9-bit mask, bit t set
  // when tap t of the pixel lies OUTSIDE the image (all set for rows past the end).  An issue
  // is then a bit extract and a shift-or: the offset with bit 31 set is past the resource's end
  // (base4 + the largest tap offset stays below 2^31), which loads zeros.
  int base4[NI];
  unsigned omask[NI];
  __device__ __forceinline__ void prepare(int row0, int wave, int lane) {
    rsrc = buffer_rsrc(x - (long long)(W + 1) * C, (uint32_t)((long long)(rows + 2 * (W + 1)) * C * 4));
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = (i * WAVES + wave) * 8 + (lane >> 3);
      const int row = row0 + r;
      const int rc = min(row, rows - 1);
      const int img = (int)fD.div(rc), p = rc - img * (int)fD.d;
      const int yy = (int)fW.div(p), xq = p - yy * W;
      const int c = DmaTile<ROWS>::swz(r, lane & 7);   // global chunk stored at lane & 7
      base4[i] = (((img * H + yy) * W + xq) * C + 4 * c) * 4;
      // opaque: the compiler would otherwise re-derive the offset from its factors at every
      // issue (a 64-bit multiply-add and three more instructions per row)
      asm volatile("" : "+v"(base4[i]));
      unsigned m = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int ky = yy + t / 3 - 1, kx = xq + t % 3 - 1;
        m |= ((unsigned)ky < (unsigned)H && (unsigned)kx < (unsigned)W) ? 0u : (1u << t);
      }
      omask[i] = row < rows ? m : 0x1FFu;
    }
  }
  template <int WV>
  __device__ __forceinline__ void issue(int k0, float* lds, int wave, int lane) const {
    static_assert(WV == WAVES, "issuer built for this workgroup shape");
    const int t = (int)fC.div(k0), cb = k0 - t * C;
    const int kh = (t * 11) >> 5, kw = t - 3 * kh;
    const uint32_t soff = (uint32_t)(((kh * W + kw) * C + cb) * 4);   // uniform, >= 0
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r0 = (i * WAVES + wave) * 8;
      const uint32_t voff = (((omask[i] >> t) & 1u) << 31) | (uint32_t)base4[i];
      buffer_dma16(rsrc, voff, soff, lds + __builtin_amdgcn_readfirstlane(r0 * DmaTile<ROWS>::BK));
    }
  }
};

template <int ROWS, int WAVES>
static DmaPatches<ROWS, WAVES> dma_patches(const float* x, int images, int H, int W, int C) {
  DmaPatches<ROWS, WAVES> d;
  d.x = x;
  d.rows = images * H * W;
  d.H = H;
  d.W = W;
  d.C = C;
  d.fD = FastDiv((uint32_t)(H * W));
  d.fW = FastDiv((uint32_t)W);
  d.fC = FastDiv((uint32_t)C);
  return d;
}

// The direct-to-LDS path needs C % 32 == 0, 16-byte aligned operands, an activation batch of
// `elems` floats (images of width W) and weight tiles within the buffer-resource span; the
// patch resource spans the batch and W + 1 pixels on either side.
static bool conv_dma_ok(const void* x, long long elems, int W, int C, const void* K) {
  return C % 32 == 0 && aligned16(x) && aligned16(K) && (elems + 2LL * (W + 1) * C) * 4 < (1LL << 31) &&
         dma_span_ok(9LL * C, 9LL * C, 256);
}

// K-outer direct-to-LDS operands of the weight-space cotangent product of one sample (k = the
// pixel p, 4 consecutive rows per 16-byte load, see DmaTileKOuter), through a buffer resource
// over the sample's tensor.  Each lane's (k-row, row chunk) inside the tile is fixed, so its row
// part is computed once per tile; pixels past D and padding taps read past the resource (zeros).
// G of the sample: rows (o, c) of O*C (C % 4 == 0), element G[o, p, c].
template <int ROWS, int WAVES, bool WHOLE = false>
struct DmaCotangentKOuter {
  using Tile = DmaTileKOuter<ROWS>;
  const float* __restrict__ g;
  int rows, D, C;
  FastDiv fC;
  static constexpr int NI = ROWS / (8 * WAVES);
  template <int WV>
  static constexpr int OPS = ROWS / (8 * WV);
  __amdgpu_buffer_rsrc_t rsrc;
  // per issued row: the byte offset of its 16-byte chunk at pixel kl (the K tile's first pixel
  // k0 adds the uniform k0 C 4 through the scalar offset), with bit 31 set for rows past the end
  // (past the resource's end: zeros), and the bound k0 < klim of the pixels inside the sample
  // (klim = D - kl), tested unless WHOLE (D a multiple of the K tile)
  int pre4[NI], klim[NI];
  __device__ __forceinline__ void prepare(int row0, int wave, int lane) {
    rsrc = buffer_rsrc(g, (uint32_t)((long long)rows * D * 4));
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int o = (i * WAVES + wave) * 256 + 4 * lane;     // float offset in the tile
      const int k = o / ROWS, pos = (o % ROWS) >> 2;
      const int row = row0 + 4 * Tile::swz(k, pos);
      const int rc = min(row, rows - 4);
      const int oo = (int)fC.div(rc), cc = rc - oo * C;
      pre4[i] = (int)((uint32_t)((oo * D * C + cc + k * C) * 4) | (row < rows ? 0u : kDmaPastEnd));
      asm volatile("" : "+v"(pre4[i]));   // kept whole, not re-derived at each issue
      klim[i] = D - k;
    }
  }
  template <int WV>
  __device__ __forceinline__ void issue(int k0, float* lds, int wave, int lane) const {
    static_assert(WV == WAVES, "issuer built for this workgroup shape");
    const uint32_t soff = (uint32_t)k0 * C * 4u;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      // WHOLE (D % 32 == 0): every pixel of every K tile is inside the sample
      const uint32_t voff = WHOLE ? (uint32_t)pre4[i] : ((uint32_t)pre4[i] | (k0 < klim[i] ? 0u : kDmaPastEnd));
      buffer_dma16(rsrc, voff, soff, lds + __builtin_amdgcn_readfirstlane((i * WAVES + wave) * 256));
    }
  }
};

// Patches of the sample's layer input [H, W, C] (C % 4 == 0): rows (tap, ci) of 9*C.
template <int ROWS, int WAVES, bool ROW32 = false>
struct DmaPatchesKOuter {
  using Tile = DmaTileKOuter<ROWS>;
  const float* __restrict__ x;
  int rows, K, H, W, C;   // K = D pixels
  FastDiv fW, fC;
  static constexpr int NI = ROWS / (8 * WAVES);
  template <int WV>
  static constexpr int OPS = ROWS / (8 * WV);
  __amdgpu_buffer_rsrc_t rsrc;
  // per issued row (tap (dy, dx), channel ci) at pixel kl of the K tile: the byte offset of its
  // shifted pixel kl + dy W + dx through a resource that starts W + 1 pixels before the sample
  // (so the offset is never negative; the K tile's first pixel k0 adds the uniform k0 C 4 through
  // the scalar offset), and what the tap's bounds test needs.  With ROW32 (W a multiple of the K
  // tile of 32 pixels) a K tile is a run of 32 pixels of one image row, and a row's tap is outside the
  // image exactly when one of the uniform conditions in its 5-bit mask `out` holds: bit 0 the
  // tile is the image's first row (dy = -1), bit 1 its last row (dy = 1), bit 2 the tile starts
  // an image row (kl = 0, dx = -1), bit 3 it ends one (kl = 31, dx = 1), bit 4 always (rows past
  // the end).
  int base4[NI], kl[NI], dy[NI], dx[NI], ok[NI];
  unsigned out[NI];
  __device__ __forceinline__ void prepare(int row0, int wave, int lane) {
    rsrc = buffer_rsrc(x - (long long)(W + 1) * C, (uint32_t)((long long)(K + W + 1) * C * 4));
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int o = (i * WAVES + wave) * 256 + 4 * lane;
      const int k = o / ROWS, pos = (o % ROWS) >> 2;
      const int row = row0 + 4 * Tile::swz(k, pos);
      const int rc = min(row, rows - 4);
      const int t = (int)fC.div(rc);
      const int kh = (t * 11) >> 5, kw = t - 3 * kh;
      const int ci = rc - t * C;
      kl[i] = k;
      dy[i] = kh - 1;
      dx[i] = kw - 1;
      base4[i] = ((k + (kh - 1) * W + (kw - 1) + W + 1) * C + ci) * 4;
      asm volatile("" : "+v"(base4[i]));   // kept whole, not re-derived at each issue
      ok[i] = row < rows ? 1 : 0;
      out[i] = (kh == 0 ? 1u : 0u) | (kh == 2 ? 2u : 0u) | (k == 0 && kw == 0 ? 4u : 0u) |
               (k == 31 && kw == 2 ? 8u : 0u) | (row < rows ? 0u : 16u);
    }
  }
  template <int WV>
  __device__ __forceinline__ void issue(int k0, float* lds, int wave, int lane) const {
    static_assert(WV == WAVES, "issuer built for this workgroup shape");
    const uint32_t soff = (uint32_t)k0 * C * 4u;
    if constexpr (ROW32) {
      const int y0 = (int)fW.div(k0), x0 = k0 - y0 * W;   // uniform
      const unsigned bad = (y0 == 0 ? 1u : 0u) | (y0 == H - 1 ? 2u : 0u) | (x0 == 0 ? 4u : 0u) |
                           (x0 + 32 == W ? 8u : 0u) | 16u;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const uint32_t voff = (uint32_t)base4[i] | ((out[i] & bad) ? kDmaPastEnd : 0u);
        buffer_dma16(rsrc, voff, soff, lds + __builtin_amdgcn_readfirstlane((i * WAVES + wave) * 256));
      }
    } else {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
      const int p = k0 + kl[i];
      const int pc = min(p, K - 1);
      const int y = (int)fW.div(pc), xx = pc - y * W;
      const bool good = ok[i] & (p < K) & ((unsigned)(y + dy[i]) < (unsigned)H) & ((unsigned)(xx + dx[i]) < (unsigned)W);
      const uint32_t voff = good ? (uint32_t)base4[i] : kDmaPastEnd;
      buffer_dma16(rsrc, voff, soff, lds + __builtin_amdgcn_readfirstlane((i * WAVES + wave) * 256));
      }
    }
  }
};

// ------------------------------------------------------------------------------ forward
template <class Cfg>
__device__ __forceinline__ void conv_fwd_epilogue(f64x4 (&acc)[Cfg::FM16][Cfg::FN16], int m0, int n0,
                                                  int M, int N, int act, const float* __restrict__ bias,
                                                  float* __restrict__ hn, float* __restrict__ dphi) {
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, double z) {
    if (bias) z += (double)bias[min(c, N - 1)];
    float h, d;
    if (act == 1) {
      h = z > 0.0 ? (float)z : 0.f;
      d = z > 0.0 ? 1.f : 0.f;
    } else {
      const float zf = (float)z;
      h = act_fwd(act, zf);
      d = act_deriv(act, zf);
    }
    if (r < M && c < N) {
      hn[(long long)r * N + c] = h;
      dphi[(long long)r * N + c] = d;
    }
  });
}

// direct-to-LDS form (C % 32 == 0): patches gathered by the DMA, three LDS stages
template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_conv_fwd_dma(DmaPatches<Cfg::BM, Cfg::WAVES> pa, DmaRowMajor<Cfg::BN, Cfg::WAVES> pb, int K, int M, int N, int act,
               const float* __restrict__ bias, float* __restrict__ hn, float* __restrict__ dphi, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f64x4 acc[Cfg::FM16][Cfg::FN16];
  zero_acc<Cfg>(acc);
  gemm_mainloop_dma_ops<Cfg, 3>(pa, pb, m0, n0, 0, K, smem, acc);
  conv_fwd_epilogue<Cfg>(acc, m0, n0, M, N, act, bias, hn, dphi);
}

template <class Cfg, bool VEC>
__global__ void __launch_bounds__(Cfg::THREADS)
k_conv_fwd(LoadPatchesKInnerT<VEC> la, LoadKInnerT<VEC> lb, int M, int N, int act,
           const float* __restrict__ bias, float* __restrict__ hn, float* __restrict__ dphi, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f64x4 acc[Cfg::FM16][Cfg::FN16];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, 0, la.K, smem, acc);
  conv_fwd_epilogue<Cfg>(acc, m0, n0, M, N, act, bias, hn, dphi);
}

template <bool VEC>
static hipError_t conv_fwd_vec(hipStream_t s, const float* x, int images, int H, int W, int Cin,
                               const float* K, int Cout, int act, const float* bias, float* hn, float* dphi) {
  using Cfg = CfgConvF64;
  using LA = LoadPatchesKInnerT<VEC>;
  using LB = LoadKInnerT<VEC>;
  LA la = patches_kinner<VEC>(x, images, H, W, Cin);
  LB lb{K, Cout, 9 * Cin, 9 * Cin};
  const int M = images * H * W;
  const int tn = cdiv(Cout, Cfg::BN), tm = cdiv(M, Cfg::BM);
  hipError_t e = set_smem<Cfg, LA, LB>((const void*)k_conv_fwd<Cfg, VEC>);
  if (e != hipSuccess) return e;
  k_conv_fwd<Cfg, VEC><<<dim3(tm * tn), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, LA, LB>(), s>>>(
      la, lb, M, Cout, act, bias, hn, dphi, tn);
  return hipGetLastError();
}

template <class Cfg>
static hipError_t conv_fwd_dma_cfg(hipStream_t s, const float* x, int images, int H, int W, int Cin,
                                   const float* K, int Cout, int act, const float* bias, float* hn, float* dphi) {
  const int M = images * H * W, Kd = 9 * Cin;
  const int tn = cdiv(Cout, Cfg::BN), tm = cdiv(M, Cfg::BM);
  auto pa = dma_patches<Cfg::BM, Cfg::WAVES>(x, images, H, W, Cin);
  DmaRowMajor<Cfg::BN, Cfg::WAVES> pb{K, Kd, Cout};
  constexpr int bytes = gemm_dma_smem_bytes<Cfg, 3>();
  hipError_t e = hipFuncSetAttribute((const void*)k_conv_fwd_dma<Cfg>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_conv_fwd_dma<Cfg><<<dim3(tm * tn), dim3(Cfg::THREADS), bytes, s>>>(pa, pb, Kd, M, Cout, act, bias, hn, dphi, tn);
  return hipGetLastError();
}

hipError_t launch_conv_fwd(hipStream_t s, const float* x, int images, int H, int W, int Cin,
                           const float* K, int Cout, int act, const float* bias, float* hn, float* dphi) {
  if (conv_dma_ok(x, (long long)images * H * W * Cin, W, Cin, K)) {
    const long long tiles = (long long)cdiv((long long)images * H * W, CfgConvF64::BM) * cdiv(Cout, CfgConvF64::BN);
    if (tiles < kConvFewTiles)
      return conv_fwd_dma_cfg<CfgConvF64Small>(s, x, images, H, W, Cin, K, Cout, act, bias, hn, dphi);
    return conv_fwd_dma_cfg<CfgConvF64>(s, x, images, H, W, Cin, K, Cout, act, bias, hn, dphi);
  }
  if (Cin % 4 == 0 && aligned16(x) && vec_ok(K, 9 * Cin, 9 * Cin))
    return conv_fwd_vec<true>(s, x, images, H, W, Cin, K, Cout, act, bias, hn, dphi);
  return conv_fwd_vec<false>(s, x, images, H, W, Cin, K, Cout, act, bias, hn, dphi);
}

// ------------------------------------------------------------------------------ GAP, seed
// g[img, c] = mean over the D pixels of h[img, p, c]: one workgroup per image.  Generic form:
// 256 threads, lanes over channels and groups of pixels; vector form (C % 4 == 0, C / 4 dividing
// 1024, 16-byte aligned): 1024 threads, a float4 of channels per lane, groups of pixels over the
// rest.  The groups' partial sums are added in a fixed order.
__global__ void __launch_bounds__(256) k_gap(const float* __restrict__ h, int D, int C, float* __restrict__ g) {
  __shared__ float part[256];
  const int img = blockIdx.x;
  const int lanes_c = C < 256 ? C : 256;
  const int groups = 256 / lanes_c;
  const int t = threadIdx.x;
  const int grp = t / lanes_c, cl = t % lanes_c;
  for (int c0 = 0; c0 < C; c0 += lanes_c) {
    const int c = c0 + cl;
    float acc = 0.f;
    if (grp < groups && c < C)
      for (int p = grp; p < D; p += groups) acc += h[((long long)img * D + p) * C + c];
    part[t] = acc;
    __syncthreads();
    if (t < lanes_c && c0 + t < C) {
      float v = 0.f;
      for (int q = 0; q < groups; ++q) v += part[q * lanes_c + t];
      g[(long long)img * C + c0 + t] = v / (float)D;
    }
    __syncthreads();
  }
}

__global__ void __launch_bounds__(1024) k_gap4(const float* __restrict__ h, int D, int C, float* __restrict__ g) {
  __shared__ float4 part[1024];
  const int img = blockIdx.x;
  const int C4 = C >> 2, groups = 1024 / C4;
  const int t = threadIdx.x, grp = t / C4, c4 = t - grp * C4;
  const float4* src = reinterpret_cast<const float4*>(h + (long long)img * D * C);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int p = grp; p < D; p += groups) {
    const float4 v = src[(long long)p * C4 + c4];
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  part[t] = acc;
  __syncthreads();
  if (t < C4) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int q = 0; q < groups; ++q) {
      const float4 w = part[q * C4 + t];
      v.x += w.x;
      v.y += w.y;
      v.z += w.z;
      v.w += w.w;
    }
    const float d = (float)D;
    float* dst = g + (long long)img * C + 4 * t;
    dst[0] = v.x / d;
    dst[1] = v.y / d;
    dst[2] = v.z / d;
    dst[3] = v.w / d;
  }
}

hipError_t launch_gap(hipStream_t s, const float* h, int images, int D, int C, float* g) {
  if (C % 4 == 0 && C / 4 <= 1024 && 1024 % (C / 4) == 0 && aligned16(h))
    k_gap4<<<dim3(images), dim3(1024), 0, s>>>(h, D, C, g);
  else
    k_gap<<<dim3(images), dim3(256), 0, s>>>(h, D, C, g);
  return hipGetLastError();
}

// G[(img*O + o), p, c] = Wd[o, c] / D * dphi[img, p, c]; blockIdx.y = img*O + o, the x-blocks
// stride over the D*C elements of that cotangent image (no 64-bit division per element).
__global__ void __launch_bounds__(256)
k_conv_seed(const float* __restrict__ Wd, const float* __restrict__ dphi, int IO, int O, int DC, FastDiv fC,
            float inv_d, float* __restrict__ G) {
  const int C = (int)fC.d;
  for (int io = blockIdx.y; io < IO; io += gridDim.y) {
    const int img = io / O, o = io - img * O;
    const float* wrow = Wd + (long long)o * C;
    const float* drow = dphi ? dphi + (long long)img * DC : nullptr;
    float* grow = G + (long long)io * DC;
    for (int q = blockIdx.x * 256 + threadIdx.x; q < DC; q += gridDim.x * 256) {
      const int c = q - (int)fC.div(q) * C;
      grow[q] = drow ? wrow[c] * inv_d * drow[q] : wrow[c] * inv_d;
    }
  }
}

// Vector form (C % 4 == 0, 16-byte aligned): workgroup w takes image w / pb and 256 float4s of
// its [D, C] plane (pixel-block w % pb); each lane loads its float4 of dphi once and writes it,
// scaled by Wd[o, c] / D, into the O cotangent images.
__global__ void __launch_bounds__(256)
k_conv_seed4(const float* __restrict__ Wd, const float* __restrict__ dphi, int images, int O, int DC4, int C4,
             float inv_d, float* __restrict__ G) {
  const int pb = (DC4 + 255) / 256;
  for (long long w = blockIdx.x; w < (long long)images * pb; w += gridDim.x) {
    const int img = (int)(w / pb);
    const int q = (int)(w - (long long)img * pb) * 256 + threadIdx.x;   // float4 index in the plane
    if (q >= DC4) continue;
    const int c4 = q % C4;
    const float4 d = dphi ? reinterpret_cast<const float4*>(dphi)[(long long)img * DC4 + q]
                          : make_float4(1.f, 1.f, 1.f, 1.f);
    for (int o = 0; o < O; ++o) {
      const float4 wv = reinterpret_cast<const float4*>(Wd)[(long long)o * C4 + c4];
      reinterpret_cast<float4*>(G)[((long long)img * O + o) * DC4 + q] =
          make_float4(wv.x * inv_d * d.x, wv.y * inv_d * d.y, wv.z * inv_d * d.z, wv.w * inv_d * d.w);
    }
  }
}

hipError_t launch_conv_seed(hipStream_t s, const float* Wd, const float* dphi, int images, int O, int D,
                            int C, float* G) {
  const int DC = D * C;
  if (C % 4 == 0 && aligned16(Wd) && aligned16(dphi) && aligned16(G)) {
    const int DC4 = DC / 4, pb = cdiv(DC4, 256);
    const long long work = (long long)images * pb;
    k_conv_seed4<<<dim3((unsigned)std::min<long long>(work, 1 << 20)), dim3(256), 0, s>>>(
        Wd, dphi, images, O, DC4, C / 4, 1.0f / (float)D, G);
    return hipGetLastError();
  }
  const int bx = std::min(cdiv(DC, 256), 64);
  const int IO = images * O;
  k_conv_seed<<<dim3(bx, std::min(IO, 32768)), dim3(256), 0, s>>>(Wd, dphi, IO, O, DC, FastDiv((uint32_t)C),
                                                                 1.0f / (float)D, G);
  return hipGetLastError();
}

// The last convolution's summand when its cotangent is the readout's (through the global pool):
// theta[n1, n2, o1, o2] += scale sum_c Wr[o1, c] Wr[o2, c] Mc[c, n1, n2].  LDS form: a workgroup
// stages Wr and w2[c][o1 O + o2] = Wr[o1, c] Wr[o2, c] once, then per block of kFoldPairs input pairs
// their Mc columns, and each thread sums entries (pair, o1, o2) from LDS.  Otherwise one thread
// per entry reads Wr and Mc directly.
constexpr int kFoldPairs = 16, kFoldIlp = 8;
constexpr int kFoldLdsFloats = 16384;
template <bool LDS>
__global__ void __launch_bounds__(256)
k_readout_fold(const float* __restrict__ Wr, int C, int O, const float* __restrict__ Mc, int N1, int N2,
               float scale, float* __restrict__ theta) {
  extern __shared__ float sm[];
  const int OO = O * O;
  const long long plane = (long long)N1 * N2;
  if (!LDS) {
    for (long long idx = blockIdx.x * 256LL + threadIdx.x; idx < plane * OO; idx += (long long)gridDim.x * 256) {
      const long long pr = idx / OO;
      const int oo = (int)(idx - pr * OO);
      const int o1 = oo / O, o2 = oo - o1 * O;
      float acc = 0.f;
      for (int c = 0; c < C; ++c) acc += (Wr[o1 * C + c] * Wr[o2 * C + c]) * Mc[c * plane + pr];
      theta[idx] += scale * acc;
    }
    return;
  }
  float* w2 = sm;
  float* mc = sm + C * OO;
  float* wr = mc + C * kFoldPairs;
  for (int i = threadIdx.x; i < O * C; i += 256) wr[i] = Wr[i];
  __syncthreads();
  for (int oo = threadIdx.x; oo < OO; oo += 256) {
    const int o1 = oo / O, o2 = oo - o1 * O;
    for (int c = 0; c < C; ++c) w2[c * OO + oo] = wr[o1 * C + c] * wr[o2 * C + c];
  }
  for (long long p0 = (long long)blockIdx.x * kFoldPairs; p0 < plane; p0 += (long long)gridDim.x * kFoldPairs) {
    const int np = (int)min<long long>(kFoldPairs, plane - p0);
    __syncthreads();   // w2 staged; the previous block's reads of mc done
    for (int i = threadIdx.x; i < C * kFoldPairs; i += 256) {
      const int c = i / kFoldPairs, j = i - c * kFoldPairs;
      mc[i] = j < np ? Mc[c * plane + p0 + j] : 0.f;
    }
    __syncthreads();
    // kFoldIlp entries per thread at once (independent sums, their LDS reads in flight together)
    const int ne = np * OO;
    for (int e0 = threadIdx.x; e0 < ne; e0 += 256 * kFoldIlp) {
      float acc[kFoldIlp];
      int wo[kFoldIlp], mo[kFoldIlp];
#pragma unroll
      for (int q = 0; q < kFoldIlp; ++q) {
        const int e = min(e0 + q * 256, ne - 1);
        const int j = e / OO;
        wo[q] = e - j * OO;
        mo[q] = j;
        acc[q] = 0.f;
      }
#pragma unroll 4
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int q = 0; q < kFoldIlp; ++q) acc[q] += w2[c * OO + wo[q]] * mc[c * kFoldPairs + mo[q]];
#pragma unroll
      for (int q = 0; q < kFoldIlp; ++q)
        if (e0 + q * 256 < ne) theta[(p0 + mo[q]) * OO + wo[q]] += scale * acc[q];
    }
  }
}

hipError_t launch_readout_fold(hipStream_t s, const float* Wr, int C, int O, const float* Mc, int N1, int N2,
                               float scale, float* theta) {
  const long long plane = (long long)N1 * N2;
  if (plane <= 0 || O <= 0 || C <= 0) return hipSuccess;
  const long long lds = (long long)C * ((long long)O * O + kFoldPairs + O);
  if (lds <= kFoldLdsFloats) {
    const unsigned grid = (unsigned)std::min<long long>((plane + kFoldPairs - 1) / kFoldPairs, 4096);
    k_readout_fold<true><<<dim3(grid), dim3(256), (size_t)lds * 4, s>>>(Wr, C, O, Mc, N1, N2, scale, theta);
  } else {
    const unsigned grid = (unsigned)std::min<long long>((plane * O * O + 255) / 256, 65536);
    k_readout_fold<false><<<dim3(grid), dim3(256), 0, s>>>(Wr, C, O, Mc, N1, N2, scale, theta);
  }
  return hipGetLastError();
}

// The batch diagonal of the folded last convolution's per-channel Grams: Mc[c][n] =
// A1[n, c, :] . A2[n, c, :] (rows of KC floats, sample n's channel c at (n C + c) KC), one wave
// per (c, n), the lanes' partial sums added in a fixed butterfly order.
__global__ void __launch_bounds__(256)
k_fold_rowdot(const float* __restrict__ A1, const float* __restrict__ A2, int n, int C, int KC,
              float* __restrict__ Mc) {
  const long long item = blockIdx.x * 4LL + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (item >= (long long)n * C) return;   // the whole wave
  const int c = (int)(item / n), i = (int)(item - (long long)c * n);
  const float* a = A1 + ((long long)i * C + c) * KC;
  const float* b = A2 + ((long long)i * C + c) * KC;
  float v = 0.f;
  for (int k = lane; k < KC; k += 64) v += a[k] * b[k];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  if (lane == 0) Mc[item] = v;
}

hipError_t launch_fold_rowdot(hipStream_t s, const float* A1, const float* A2, int n, int C, int KC, float* Mc) {
  const long long items = (long long)n * C;
  if (items <= 0) return hipSuccess;
  if ((items + 3) / 4 > 0x7fffffffLL) return hipErrorInvalidValue;
  k_fold_rowdot<<<dim3((unsigned)((items + 3) / 4)), dim3(256), 0, s>>>(A1, A2, n, C, KC, Mc);
  return hipGetLastError();
}

// The traced output of the folded last convolution: theta[n1, n2] += scale sum_c w_c Mc[c][n1, n2]
// with w_c = sum_o Wr[o, c]^2 (the trace of Wr[o1, c] Wr[o2, c] over o), staged in LDS when the C
// weights fit (LDS), else formed per channel from Wr; one pair per thread, channels in order.
template <bool LDS>
__global__ void __launch_bounds__(256)
k_readout_fold_trace(const float* __restrict__ Wr, int C, int O, const float* __restrict__ Mc, long long plane,
                     float scale, float* __restrict__ theta) {
  extern __shared__ float wsum[];
  auto weight = [&](int c) -> float {
    float v = 0.f;
    for (int o = 0; o < O; ++o) {
      const float x = Wr[(long long)o * C + c];
      v += x * x;
    }
    return v;
  };
  if (LDS) {
    for (int c = threadIdx.x; c < C; c += 256) wsum[c] = weight(c);
    __syncthreads();
  }
  for (long long p = blockIdx.x * 256LL + threadIdx.x; p < plane; p += (long long)gridDim.x * 256) {
    float acc = 0.f;
    for (int c = 0; c < C; ++c) acc += (LDS ? wsum[c] : weight(c)) * Mc[(long long)c * plane + p];
    theta[p] += scale * acc;
  }
}

hipError_t launch_readout_fold_trace(hipStream_t s, const float* Wr, int C, int O, const float* Mc, int N1, int N2,
                                     float scale, float* theta) {
  const long long plane = (long long)N1 * N2;
  if (plane <= 0 || O <= 0 || C <= 0) return hipSuccess;
  const unsigned grid = (unsigned)std::min<long long>((plane + 255) / 256, 4096);
  if (C <= kFoldLdsFloats)
    k_readout_fold_trace<true><<<dim3(grid), dim3(256), (size_t)C * 4, s>>>(Wr, C, O, Mc, plane, scale, theta);
  else
    k_readout_fold_trace<false><<<dim3(grid), dim3(256), 0, s>>>(Wr, C, O, Mc, plane, scale, theta);
  return hipGetLastError();
}

// Kt[ci, kh, kw, co] = K[co, 2 - kh, 2 - kw, ci]
__global__ void k_conv_flip(const float* __restrict__ K, int Cout, int Cin, float* __restrict__ Kt) {
  const int total = Cout * 9 * Cin;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int co = i % Cout;
    const int rest = i / Cout;
    const int tap = rest % 9, ci = rest / 9;
    const int kh = tap / 3, kw = tap % 3;
    Kt[i] = K[((co * 3 + (2 - kh)) * 3 + (2 - kw)) * Cin + ci];
  }
}

hipError_t launch_conv_flip(hipStream_t s, const float* K, int Cout, int Cin, float* Kt) {
  const int total = Cout * 9 * Cin;
  k_conv_flip<<<dim3(cdiv(total, 256)), dim3(256), 0, s>>>(K, Cout, Cin, Kt);
  return hipGetLastError();
}

// Kernel z of the batch: blockIdx.y; tap t of T is read from tap T - 1 - t (the 3x3 flip:
// (kh, kw) -> (2 - kh, 2 - kw); with T = 1 a transpose).
__global__ void __launch_bounds__(256) k_conv_flip_batch(FlipBatch b) {
  const int z = blockIdx.y;
  const int Cout = b.Cout[z], Cin = b.Cin[z], T = b.taps[z];
  const int total = Cout * T * Cin;
  const float* __restrict__ K = b.K[z];
  float* __restrict__ Kt = b.Kt[z];
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int co = i % Cout;
    const int rest = i / Cout;
    const int tap = rest % T, ci = rest / T;
    Kt[i] = K[((long long)co * T + (T - 1 - tap)) * Cin + ci];
  }
}

hipError_t launch_conv_flip_batch(hipStream_t s, const FlipBatch& b) {
  if (b.count <= 0) return hipSuccess;
  if (b.count > kMaxLayers) return hipErrorInvalidValue;
  long long most = 0;
  for (int z = 0; z < b.count; ++z) {
    if (b.taps[z] != 1 && b.taps[z] != 9) return hipErrorInvalidValue;
    most = std::max(most, (long long)b.Cout[z] * b.taps[z] * b.Cin[z]);
  }
  if (most >= (1LL << 31)) return hipErrorInvalidValue;
  k_conv_flip_batch<<<dim3((unsigned)std::min<long long>(cdiv(most, 256), 1024), b.count), dim3(256), 0, s>>>(b);
  return hipGetLastError();
}

// J[(s*O + o), off + c*KCs + js] = acc[r = o*C + c, k] for the GEMM columns k of KC = F Cin
// (F taps of Cin computed input channels), stored as the columns js of KCs = F Cst (the first Cst
// channels of each tap: a layer input padded from Cst to Cin channels has zero columns that are
// not stored; Cst = Cin: js = k).  A fragment inside R = O*C and inside one o (no multiple of C
// in (r0, r0 + 31]) writes 32 consecutive c of one row of J, addressed from one base (32-bit byte
// offsets: KCs < 2^25).
template <class Cfg>
__device__ __forceinline__ void conv_wgrad_store(f32x16 (&acc)[Cfg::FM][Cfg::FN], int m0, int n0, int s,
                                                 int O, FastDiv fC, int KC, FastDiv fCin, int Cst,
                                                 float* __restrict__ J, long long ldJ, long long off) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
  const int C = (int)fC.d, R = O * C;
  const int Cin = (int)fCin.d, KCs = Cst == Cin ? KC : (KC / Cin) * Cst;
  // the stored column of GEMM column k, or -1 (a padded channel or past KC)
  auto col = [&](int k) {
    if (k >= KC) return -1;
    if (Cst == Cin) return k;
    const int tap = (int)fCin.div(k), ci = k - tap * Cin;
    return ci < Cst ? tap * Cst + ci : -1;
  };
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm) {
    const int r0 = __builtin_amdgcn_readfirstlane(m0 + wm0 + fm * 32);
    if (r0 >= R) continue;
    const int o0 = (int)fC.div(r0);
    if (r0 + 32 <= R && KCs < (1 << 25) && (int)fC.div(r0 + 31) == o0) {
      float* base = J + ((long long)s * O + o0) * ldJ + off + (long long)(r0 - o0 * C) * KCs;
#pragma unroll
      for (int fn = 0; fn < Cfg::FN; ++fn) {
        const int js = col(n0 + wn0 + fn * 32 + (lane & 31));
        if (js < 0) continue;
#pragma unroll
        for (int v = 0; v < 16; ++v) at_bytes(base, (uint32_t)(frag_row(v, lane) * KCs + js) * 4u) = acc[fm][fn][v];
      }
    } else {
#pragma unroll
      for (int fn = 0; fn < Cfg::FN; ++fn) {
        const int js = col(n0 + wn0 + fn * 32 + (lane & 31));
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = r0 + frag_row(v, lane);
          if (r < R && js >= 0) {
            const int o = (int)fC.div(r), c = r - o * C;
            J[((long long)s * O + o) * ldJ + off + (long long)c * KCs + js] = acc[fm][fn][v];
          }
        }
      }
    }
  }
}
// out[(img*O+o), p, ci] = (sum_k patch(G)[.., p, k] Kt[ci, k]) * dphi[img, p, ci]
template <class Cfg, bool VEC>
__global__ void __launch_bounds__(Cfg::THREADS)
k_conv_bwd(LoadPatchesKInnerT<VEC> la, LoadKInnerT<VEC> lb, const float* __restrict__ dphi, int R,
           int N, FastDiv fOD, FastDiv fD, float* __restrict__ out, int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, 0, la.K, smem, acc);
  store_pixel_rows<Cfg>(acc, m0, n0, dphi, out, R, N, fOD, fD);
}

// direct-to-LDS form (Cg % 32 == 0): the cotangent patches gathered by the DMA, NS LDS stages
template <class Cfg, int NS>
__global__ void __launch_bounds__(Cfg::THREADS)
k_conv_bwd_dma(DmaPatches<Cfg::BM, Cfg::WAVES> pa, DmaRowMajor<Cfg::BN, Cfg::WAVES> pb, int K,
               const float* __restrict__ dphi, int R, int N, FastDiv fOD, FastDiv fD, float* __restrict__ out,
               int tiles_n) {
  extern __shared__ float smem[];
  const int tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  gemm_mainloop_dma_ops<Cfg, NS>(pa, pb, m0, n0, 0, K, smem, acc);
  store_pixel_rows<Cfg>(acc, m0, n0, dphi, out, R, N, fOD, fD);
}

template <bool VEC>
static hipError_t conv_bwd_vec(hipStream_t s, const float* G, int images, int O, int H, int W, int Cg,
                               const float* Kt, int Cin, const float* dphi, float* out) {
  using Cfg = CfgConv;
  using LA = LoadPatchesKInnerT<VEC>;
  using LB = LoadKInnerT<VEC>;
  const int D = H * W;
  LA la = patches_kinner<VEC>(G, images * O, H, W, Cg);
  LB lb{Kt, Cin, 9 * Cg, 9 * Cg};
  int R;
  if (!to_int((long long)images * O * D, R)) return hipErrorInvalidValue;
  const int tn = cdiv(Cin, Cfg::BN), tm = cdiv(R, Cfg::BM);
  hipError_t e = set_smem<Cfg, LA, LB>((const void*)k_conv_bwd<Cfg, VEC>);
  if (e != hipSuccess) return e;
  k_conv_bwd<Cfg, VEC><<<dim3(tm * tn), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, LA, LB>(), s>>>(
      la, lb, dphi, R, Cin, FastDiv((uint32_t)(O * D)), FastDiv((uint32_t)D), out, tn);
  return hipGetLastError();
}

template <class Cfg>
static hipError_t conv_bwd_dma_cfg(hipStream_t s, const float* G, int images, int O, int H, int W, int Cg,
                                   const float* Kt, int Cin, const float* dphi, float* out) {
  constexpr int NS = kConvBwdStages;
  const int D = H * W, Kd = 9 * Cg;
  int R;
  if (!to_int((long long)images * O * D, R)) return hipErrorInvalidValue;
  const int tn = cdiv(Cin, Cfg::BN), tm = cdiv(R, Cfg::BM);
  auto pa = dma_patches<Cfg::BM, Cfg::WAVES>(G, images * O, H, W, Cg);
  DmaRowMajor<Cfg::BN, Cfg::WAVES> pb{Kt, Kd, Cin};
  constexpr int bytes = gemm_dma_smem_bytes<Cfg, NS>();
  hipError_t e = hipFuncSetAttribute((const void*)k_conv_bwd_dma<Cfg, NS>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  k_conv_bwd_dma<Cfg, NS><<<dim3(tm * tn), dim3(Cfg::THREADS), bytes, s>>>(
      pa, pb, Kd, dphi, R, Cin, FastDiv((uint32_t)(O * D)), FastDiv((uint32_t)D), out, tn);
  return hipGetLastError();
}

hipError_t launch_conv_bwd(hipStream_t s, const float* G, int images, int O, int H, int W, int Cg,
                           const float* Kt, int Cin, const float* dphi, float* out) {
  if (conv_dma_ok(G, (long long)images * O * H * W * Cg, W, Cg, Kt)) {
    const long long tiles = (long long)cdiv((long long)images * O * H * W, CfgConvBwd::BM) * cdiv(Cin, CfgConvBwd::BN);
    if (tiles < kConvFewTiles) return conv_bwd_dma_cfg<CfgConv>(s, G, images, O, H, W, Cg, Kt, Cin, dphi, out);
    return conv_bwd_dma_cfg<CfgConvBwd>(s, G, images, O, H, W, Cg, Kt, Cin, dphi, out);
  }
  if (Cg % 4 == 0 && aligned16(G) && vec_ok(Kt, 9 * Cg, 9 * Cg))
    return conv_bwd_vec<true>(s, G, images, O, H, W, Cg, Kt, Cin, dphi, out);
  return conv_bwd_vec<false>(s, G, images, O, H, W, Cg, Kt, Cin, dphi, out);
}

// ------------------------------------------------------------------------------ weight-space cotangent
// For sample s = blockIdx.y:  J[s*O + o][off + c*KC + k] = sum_p G[s,o,p,c] patch[s,p,k]
// (VA / VB: float4 loads of the cotangent / patch operand)
template <class Cfg, bool VA, bool VB, bool PW>
__global__ void __launch_bounds__(Cfg::THREADS)
k_conv_wgrad(const float* __restrict__ G, const float* __restrict__ h, int O, int H, int W, int C,
             int Cin, FastDiv fC, FastDiv fW, FastDiv fCin, float* __restrict__ J, long long ldJ,
             long long off, int tiles_m, int tiles_n, int samples) {
  extern __shared__ float smem[];
  int s, t;
  if (!xcd_sample_tile(blockIdx.x, tiles_m * tiles_n, samples, s, t)) return;
  const int D = H * W;
  const int KC = PW ? Cin : 9 * Cin;
  const int tm = t / tiles_n, tn = t - tm * tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  LoadCotangentKOuterT<VA> la;
  la.g = G + (long long)s * O * D * C;
  la.rows = O * C;
  la.K = D;
  la.C = C;
  la.D = D;
  la.fC = fC;
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  if constexpr (PW) {
    // pointwise: the columns are the input channels themselves, [D, Cin] of the sample
    LoadCotangentKOuterT<VB> lb;
    lb.g = h + (long long)s * D * Cin;
    lb.rows = Cin;
    lb.K = D;
    lb.C = Cin;
    lb.D = D;
    lb.fC = fCin;
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, D, smem, acc);
  } else {
    LoadPatchesKOuterT<VB> lb;
    lb.x = h + (long long)s * D * Cin;
    lb.rows = KC;
    lb.K = D;
    lb.H = H;
    lb.W = W;
    lb.C = Cin;
    lb.fW = fW;
    lb.fC = fCin;
    gemm_mainloop<Cfg>(la, lb, m0, n0, 0, D, smem, acc);
  }
  conv_wgrad_store<Cfg>(acc, m0, n0, s, O, fC, KC, fCin, Cin, J, ldJ, off);
}

// direct-to-LDS form (C % 4 == 0 and Cin % 4 == 0): both operands K-outer, NS LDS stages
// AL: every K tile of 32 pixels is whole (D % 32 == 0) and, for the 3x3 patches, lies in one
// image row (W % 32 == 0)
template <class Cfg, int NS, bool PW, bool AL>
__global__ void __launch_bounds__(Cfg::THREADS)
k_conv_wgrad_dma(const float* __restrict__ G, const float* __restrict__ h, int O, int H, int W, int C, int Cin, FastDiv fC, FastDiv fW, FastDiv fCin,
                 int Cst, float* __restrict__ J, long long ldJ, long long off, int tiles_m, int tiles_n, int samples) {
  extern __shared__ float smem[];
  int s, t;
  if (!xcd_sample_tile(blockIdx.x, tiles_m * tiles_n, samples, s, t)) return;
  const int D = H * W;
  const int KC = PW ? Cin : 9 * Cin;
  const int tm = t / tiles_n, tn = t - tm * tiles_n;
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  DmaCotangentKOuter<Cfg::BM, Cfg::WAVES, AL> ia;
  ia.g = G + (long long)s * O * D * C;
  ia.rows = O * C;
  ia.D = D;
  ia.C = C;
  ia.fC = fC;
  // two MFMA chains per fragment (DualAcc), added after the K loop
  DualAcc dacc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) dacc[fm][fn].v[0][v] = dacc[fm][fn].v[1][v] = 0.f;
  if constexpr (PW) {
    // pointwise: the columns are the input channels themselves, [D, Cin] of the sample
    DmaCotangentKOuter<Cfg::BN, Cfg::WAVES, AL> ib;
    ib.g = h + (long long)s * D * Cin;
    ib.rows = Cin;
    ib.D = D;
    ib.C = Cin;
    ib.fC = fCin;
    gemm_mainloop_dma_ops<Cfg, NS>(ia, ib, m0, n0, 0, D, smem, dacc);
  } else {
    DmaPatchesKOuter<Cfg::BN, Cfg::WAVES, AL> ib;
    ib.x = h + (long long)s * D * Cin;
    ib.rows = KC;
    ib.K = D;
    ib.H = H;
    ib.W = W;
    ib.C = Cin;
    ib.fW = fW;
    ib.fC = fCin;
    gemm_mainloop_dma_ops<Cfg, NS>(ia, ib, m0, n0, 0, D, smem, dacc);
  }
  f32x16 acc[Cfg::FM][Cfg::FN];
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn) acc[fm][fn] = dacc[fm][fn].v[0] + dacc[fm][fn].v[1];
  conv_wgrad_store<Cfg>(acc, m0, n0, s, O, fC, KC, fCin, Cst, J, ldJ, off);
}

// Grid of the per-sample weight-space products: the tiles of one sample on one XCD, so the
// column tiles that share a block of cotangent rows (and the row tiles that share the patch
// columns) read them through one L2 (xcd_sample_tile).
static unsigned wgrad_grid(int tiles, int images) { return (unsigned)(8 * ((images + 7) / 8) * tiles); }

template <bool VA, bool VB, bool PW>
static hipError_t conv_wgrad_vec(hipStream_t s, const float* G, const float* h, int images, int O,
                                 int H, int W, int C, int Cin, float* J, long long ldJ, long long off) {
  using Cfg = CfgConv;
  using LA = LoadCotangentKOuterT<VA>;
  using LB = std::conditional_t<PW, LoadCotangentKOuterT<VB>, LoadPatchesKOuterT<VB>>;
  const int tn = cdiv((PW ? 1 : 9) * Cin, Cfg::BN), tm = cdiv(O * C, Cfg::BM);
  hipError_t e = set_smem<Cfg, LA, LB>((const void*)k_conv_wgrad<Cfg, VA, VB, PW>);
  if (e != hipSuccess) return e;
  k_conv_wgrad<Cfg, VA, VB, PW><<<dim3(wgrad_grid(tm * tn, images)), dim3(Cfg::THREADS),
                                  gemm_smem_bytes<Cfg, LA, LB>(), s>>>(
      G, h, O, H, W, C, Cin, FastDiv((uint32_t)C), FastDiv((uint32_t)W), FastDiv((uint32_t)Cin), J,
      ldJ, off, tm, tn, images);
  return hipGetLastError();
}

// Per-sample weight-space product of a 3x3 (PW = false: columns (tap, ci) of the patches) or a
// pointwise (PW = true: columns ci of the layer input) convolution.
template <bool PW>
static hipError_t conv_wgrad_any(hipStream_t s, const float* G, const float* h, int images, int O, int H,
                                 int W, int C, int Cin, float* J, long long ldJ, long long off, int Cst) {
  const int KC = (PW ? 1 : 9) * Cin;
  if ((long long)8 * ((images + 7) / 8) * cdiv(KC, CfgConv::BN) * cdiv((long long)O * C, CfgConv::BM) >=
      (1LL << 31))
    return hipErrorInvalidValue;
  // direct-to-LDS: one sample's cotangents and layer input each within a buffer resource
  if (C % 4 == 0 && Cin % 4 == 0 && aligned16(G) && aligned16(h) && (long long)O * H * W * C * 4 < (1LL << 31) &&
      (long long)H * W * Cin * 4 < (1LL << 31)) {
    constexpr int NS = kConvWgStages;
    auto go = [&](auto cfg_tag, auto al_tag) -> hipError_t {
      using Cfg = decltype(cfg_tag);
      constexpr bool AL = decltype(al_tag)::value;
      const int tn = cdiv(KC, Cfg::BN), tm = cdiv(O * C, Cfg::BM);
      constexpr int bytes = gemm_dma_smem_bytes<Cfg, NS>();
      hipError_t e = hipFuncSetAttribute((const void*)k_conv_wgrad_dma<Cfg, NS, PW, AL>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
      if (e != hipSuccess) return e;
      k_conv_wgrad_dma<Cfg, NS, PW, AL><<<dim3(wgrad_grid(tm * tn, images)), dim3(Cfg::THREADS), bytes, s>>>(
          G, h, O, H, W, C, Cin, FastDiv((uint32_t)C), FastDiv((uint32_t)W), FastDiv((uint32_t)Cin), Cst, J,
          ldJ, off, tm, tn, images);
      return hipGetLastError();
    };
    const bool al = PW ? (H * W) % 32 == 0 : W % 32 == 0;
    // at most 64 rows (O C: one output, as for the folded last convolution): 64 x 64 tiles
    if (O * C <= 64)
      return al ? go(CfgConvWgSmall{}, std::true_type{}) : go(CfgConvWgSmall{}, std::false_type{});
    return al ? go(CfgConvWg{}, std::true_type{}) : go(CfgConvWg{}, std::false_type{});
  }
  if (Cst != Cin) return hipErrorInvalidValue;   // padded inputs take the direct-to-LDS form only
  const bool va = C % 4 == 0 && aligned16(G), vb = Cin % 4 == 0 && aligned16(h);
  if (va && vb) return conv_wgrad_vec<true, true, PW>(s, G, h, images, O, H, W, C, Cin, J, ldJ, off);
  if (va) return conv_wgrad_vec<true, false, PW>(s, G, h, images, O, H, W, C, Cin, J, ldJ, off);
  return conv_wgrad_vec<false, false, PW>(s, G, h, images, O, H, W, C, Cin, J, ldJ, off);
}

hipError_t launch_conv_wgrad(hipStream_t s, const float* G, const float* h, int images, int O, int H,
                             int W, int C, int Cin, float* J, long long ldJ, long long off) {
  return conv_wgrad_any<false>(s, G, h, images, O, H, W, C, Cin, J, ldJ, off, Cin);
}

hipError_t launch_pw_wgrad(hipStream_t s, const float* G, const float* h, int images, int O, int H, int W,
                           int C, int Cin, float* J, long long ldJ, long long off) {
  return conv_wgrad_any<true>(s, G, h, images, O, H, W, C, Cin, J, ldJ, off, Cin);
}

// xp [rows, Cp] = x [rows, Cin] with zero channels Cin .. Cp - 1.
__global__ void __launch_bounds__(256)
k_pad_channels(const float* __restrict__ x, long long rows, int Cin, int Cp, float* __restrict__ xp) {
  const long long total = rows * Cp;
  for (long long i = blockIdx.x * 256LL + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const long long r = i / Cp;
    const int c = (int)(i - r * Cp);
    xp[i] = c < Cin ? x[r * Cin + c] : 0.f;
  }
}

// (images of fewer than kPadMinPixels pixels keep the register-staged form: a few K tiles per
// sample do not repay the copy; 4x4 images measured slower padded)
constexpr int kPadMinPixels = 256;
bool conv_wgrad_pad_ok(int images, int O, int H, int W, int C, int Cin, const float* G, const float* xp) {
  const int Cp = (Cin + 3) & ~3;
  return Cin % 4 != 0 && C % 4 == 0 && H * W >= kPadMinPixels && aligned16(G) && aligned16(xp) &&
         (long long)O * H * W * C * 4 < (1LL << 31) && (long long)H * W * Cp * 4 < (1LL << 31) &&
         (long long)images * H * W * Cp < (1LL << 40);
}

hipError_t launch_conv_wgrad_padded(hipStream_t s, const float* G, const float* h, float* xp, int images, int O,
                                    int H, int W, int C, int Cin, float* J, long long ldJ, long long off, bool pw) {
  const int Cp = (Cin + 3) & ~3;
  if (!conv_wgrad_pad_ok(images, O, H, W, C, Cin, G, xp)) return hipErrorInvalidValue;
  const long long rows = (long long)images * H * W;
  k_pad_channels<<<dim3((unsigned)std::min<long long>((rows * Cp + 255) / 256, 16384)), dim3(256), 0, s>>>(
      h, rows, Cin, Cp, xp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return pw ? conv_wgrad_any<true>(s, G, xp, images, O, H, W, C, Cp, J, ldJ, off, Cin)
            : conv_wgrad_any<false>(s, G, xp, images, O, H, W, C, Cp, J, ldJ, off, Cin);
}

// ------------------------------------------------------------------------------ split-K J1 J2^T
__device__ __forceinline__ void tri_index_c(int t, int nt, int& tm, int& tn) {
  int r = 0, base = 0;
  while (base + (nt - r) <= t) {
    base += nt - r;
    ++r;
  }
  tm = r;
  tn = r + (t - base);
}

// part[z][r1][r2] = sum_{k in chunk z} J1[r1, k] J2[r2, k]
template <class Cfg, bool VEC>
__global__ void __launch_bounds__(Cfg::THREADS)
k_ntk_splitk(LoadKInnerT<VEC> la, LoadKInnerT<VEC> lb, int chunk, int symmetric, float* __restrict__ part,
             int tiles_n) {
  extern __shared__ float smem[];
  const int z = blockIdx.y;
  int tm, tn;
  if (symmetric) {
    tri_index_c(blockIdx.x, tiles_n, tm, tn);
  } else {
    tm = blockIdx.x / tiles_n;
    tn = blockIdx.x % tiles_n;
  }
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int k0 = z * chunk;
  const int k1 = min(la.K, k0 + chunk);
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  gemm_mainloop<Cfg>(la, lb, m0, n0, k0, k1, smem, acc);
  const int R1 = la.rows, R2 = lb.rows;
  float* P = part + (long long)z * R1 * R2;
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, float v) {
    if (r < R1 && c < R2) P[(long long)r * R2 + c] = v;
  });
}

// Direct-to-LDS form (K-contiguous 16-byte aligned rows, K % 32 == 0): the same products, with
// the work items ordered per XCD.  The items (chunk z, tile t) are numbered chunk by chunk,
// i = z * tiles + t, and cut into 8 equal contiguous ranges, one per XCD.  Workgroup b runs on
// XCD x = b % 8 (the hardware hands out workgroup ids round robin over the 8 XCDs) and takes
// the (b / 8)-th item of range x, so the tiles of a chunk run together on one XCD and share its
// L2 for the rows of J1 and J2 they read.
template <class Cfg>
__global__ void __launch_bounds__(Cfg::THREADS)
k_ntk_splitk_dma(const float* __restrict__ J1, const float* __restrict__ J2, int R1, int R2, int K,
                 long long ld, int chunk, int splits, int tiles, int symmetric, float* __restrict__ part,
                 int tiles_n) {
  extern __shared__ float smem[];
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const long long items = (long long)tiles * splits;
  const long long i = x * items / 8 + j;
  if (i >= (x + 1) * items / 8) return;
  const int z = (int)(i / tiles), t = (int)(i - (long long)z * tiles);
  int tm, tn;
  if (symmetric) {
    tri_index_c(t, tiles_n, tm, tn);
  } else {
    tm = t / tiles_n;
    tn = t % tiles_n;
  }
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int k0 = z * chunk;
  const int k1 = min(K, k0 + chunk);
  f32x16 acc[Cfg::FM][Cfg::FN];
  zero_acc<Cfg>(acc);
  gemm_mainloop_dma<Cfg, 2>(J1, ld, R1, J2, ld, R2, m0, n0, k0, k1, smem, acc);
  float* P = part + (long long)z * R1 * R2;
  for_each_acc<Cfg>(acc, m0, n0, [&](int r, int c, float v) {
    if (r < R1 && c < R2) P[(long long)r * R2 + c] = v;
  });
}

// theta[n1][n2][o1][o2] = w[n1, n2] sum_z part[z][r1][r2] + (o1 == o2) rscale gram[n1, n2], or,
// with accumulate, theta += w[n1, n2] sum_z part[z][r1][r2] (the readout summand is then
// already in theta).  w = null means 1; gram = null means no readout summand.
__global__ void k_ntk_reduce(const float* __restrict__ part, int splits, int N1, int N2, int O,
                             int symmetric, int tile, const float* __restrict__ w,
                             const float* __restrict__ gram, float rscale, int accumulate,
                             float* __restrict__ theta) {
  const int R1 = N1 * O, R2 = N2 * O;   // below 2^31: the launcher checked them
  const long long total = (long long)R1 * R2;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int r1 = (int)(i / R2), r2 = (int)(i - (long long)r1 * R2);
    long long src = i;
    if (symmetric && (r1 / tile) > (r2 / tile)) src = (long long)r2 * R2 + r1;
    float a[4] = {0.f, 0.f, 0.f, 0.f};   // four independent chains keep several loads in flight
    int z = 0;
    for (; z + 4 <= splits; z += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] += part[(long long)(z + u) * total + src];
    }
    for (; z < splits; ++z) a[0] += part[(long long)z * total + src];
    float v = (a[0] + a[1]) + (a[2] + a[3]);
    const int n1 = r1 / O, o1 = r1 - n1 * O, n2 = r2 / O, o2 = r2 - n2 * O;
    if (w) v *= w[(long long)n1 * N2 + n2];
    float* dst = theta + (((long long)n1 * N2 + n2) * O + o1) * O + o2;
    if (accumulate)
      v += *dst;
    else if (o1 == o2 && gram)
      v += rscale * gram[(long long)n1 * N2 + n2];
    *dst = v;
  }
}

int splitk_tile() { return CfgSplitK::BM; }

int splitk_plan(int R1, int R2, long long K, int symmetric, long long part_capacity, int* chunk_out) {
  using Cfg = CfgSplitK;
  const int tm = cdiv(R1, Cfg::BM), tn = cdiv(R2, Cfg::BN);
  const int tiles = symmetric ? tn * (tn + 1) / 2 : tm * tn;
  // aim for about 4 workgroups per compute unit, with chunks that are whole K tiles, and
  // never more partial [R1, R2] products than the workspace holds
  long long want = std::min<long long>(1024 / std::max(tiles, 1), cdiv(K, 256));
  want = std::min<long long>(want, part_capacity / ((long long)R1 * R2));
  int splits = (int)std::max<long long>(1, want);
  long long chunk = (K + splits - 1) / splits;
  chunk = ((chunk + Cfg::BK - 1) / Cfg::BK) * Cfg::BK;
  splits = (int)((K + chunk - 1) / chunk);
  *chunk_out = (int)chunk;
  return splits;
}

template <bool VEC>
static hipError_t splitk_vec(hipStream_t s, const float* J1, const float* J2, int R1, int R2,
                             long long K, long long ld, int symmetric, int chunk, int splits,
                             float* part) {
  using Cfg = CfgSplitK;
  using L = LoadKInnerT<VEC>;
  L la{J1, R1, (int)K, ld};
  L lb{J2, R2, (int)K, ld};
  const int tm = cdiv(R1, Cfg::BM), tn = cdiv(R2, Cfg::BN);
  const int tiles = symmetric ? tn * (tn + 1) / 2 : tm * tn;
  hipError_t e = set_smem<Cfg, L, L>((const void*)k_ntk_splitk<Cfg, VEC>);
  if (e != hipSuccess) return e;
  k_ntk_splitk<Cfg, VEC><<<dim3(tiles, splits), dim3(Cfg::THREADS), gemm_smem_bytes<Cfg, L, L>(), s>>>(
      la, lb, chunk, symmetric, part, tn);
  return hipGetLastError();
}

hipError_t launch_ntk_splitk(hipStream_t s, const float* J1, const float* J2, int R1, int R2,
                             long long K, long long ld, int symmetric, int chunk, int splits,
                             float* part) {
  if (vec_ok(J1, ld, K) && vec_ok(J2, ld, K) && K % 32 == 0 && chunk % 32 == 0 && dma_span_ok(ld, K, 128)) {
    using Cfg = CfgSplitKDma;
    static_assert(Cfg::BM == CfgSplitK::BM && Cfg::BN == CfgSplitK::BN, "the reduction's tile grid");
    const int tm = cdiv(R1, Cfg::BM), tn = cdiv(R2, Cfg::BN);
    const int tiles = symmetric ? tn * (tn + 1) / 2 : tm * tn;
    constexpr int bytes = gemm_dma_smem_bytes<Cfg, 2>();
    hipError_t e = hipFuncSetAttribute((const void*)k_ntk_splitk_dma<Cfg>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    const long long blocks = 8 * (((long long)tiles * splits + 7) / 8);
    k_ntk_splitk_dma<Cfg><<<dim3((unsigned)blocks), dim3(Cfg::THREADS), bytes, s>>>(
        J1, J2, R1, R2, (int)K, ld, chunk, splits, tiles, symmetric, part, tn);
    return hipGetLastError();
  }
  if (vec_ok(J1, ld, K) && vec_ok(J2, ld, K))
    return splitk_vec<true>(s, J1, J2, R1, R2, K, ld, symmetric, chunk, splits, part);
  return splitk_vec<false>(s, J1, J2, R1, R2, K, ld, symmetric, chunk, splits, part);
}

hipError_t launch_ntk_reduce(hipStream_t s, const float* part, int splits, int N1, int N2, int O,
                             int symmetric, const float* w, const float* gram, float rscale,
                             int accumulate, float* theta) {
  int R1, R2;
  if (!to_int((long long)N1 * O, R1) || !to_int((long long)N2 * O, R2)) return hipErrorInvalidValue;
  const long long total = (long long)R1 * R2;
  const int blocks = (int)std::min<long long>((total + 255) / 256, 256 * 64);
  k_ntk_reduce<<<dim3(blocks), dim3(256), 0, s>>>(part, splits, N1, N2, O, symmetric, CfgSplitK::BM,
                                                  w, gram, rscale, accumulate, theta);
  return hipGetLastError();
}

}  // namespace ntk
