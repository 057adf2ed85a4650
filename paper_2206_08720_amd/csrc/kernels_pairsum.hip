// kernels_pairsum.hip -- the inside-out contraction order of a convolution's NTK summand, on the
// matrix cores (appendix "CNN NTK Complexity", Table complexities_cnn: the inside-out order,
// N^2 (D^2 F W + O D^2 W + O^2 D W) multiply-adds).
//
// For a 3x3 SAME convolution (F = 9 taps) or a pointwise one (F = 1) with input h [M, D, Cin] and
// output cotangent G [M*O, D, C] (the stacked batch), and every input pair (n1, n2):
//   H[q1, q2]    = h1[q1] . h2[q2]                           the pixel Gram (K = Cin)
//   PK[p1, p2]   = sum over the taps t of H[p1 + t, p2 + t]   the patch-pair Gram: both patches take
//                  (both shifted pixels inside the image)     the same tap (F = 1: PK = H)
//   X[o1, c, p2] = sum_p1 G1[o1, p1, c] PK[p1, p2]
//   theta[o1, o2] (+)= sum_{c, p2} X[o1, c, p2] G2[o2, p2, c]
// i.e. the sum over pixel pairs of (patch1 . patch2) times the cotangent product, with the
// channel sum taken inside.  The readout summand (g1 . g2) delta_{o1 o2} is added by the call
// that writes theta first.
//
// Matrix-core form (v_mfma_f32_16x16x4_f32; lane l of a wave, g = l / 16, i = l % 16):
//   A: lane l supplies A[i][g];  B: lane l supplies B[g][i];  D: lane l, register v holds D[4g+v][i].
// Each wave takes one input pair, or four sharing their batch-1 sample (PairGeom):
//   * H in 16 x 16 blocks, K = Cin in steps of 16 (the j-th MFMA of a step takes ci = k0 + 4g + j),
//     staged in LDS; each lane then forms in registers the PK entries it supplies as A operands,
//     pk[rt][t][j] = PK[16t + 4g + j][16rt + i].
//   * Per channel c and block rt of 16 pixels p2:
//       X^T[p2][o1] = sum_p1 PK[p1][p2] G1[c][o1][p1]     A = pk, B = G1 (one 16-byte LDS read per t)
//     and the accumulator of that product is the A operand of
//       theta[o1][o2] += sum_p2 X^T[p2][o1] G2[c][o2][p2]  (the v-th MFMA takes p2 = 16rt + 4g + v)
//     so X never leaves the registers.
// The output rows o1 and columns o2 come in blocks of 16 (O padded with zero cotangent rows);
// pixels are padded to Dp = 16 DT with zero PK entries.  The cotangent is read from a copy laid
// out [M, C, O, Dp] (k_pair_gt), staged through LDS per chunk of channels for the block of input
// pairs of a workgroup (PairGeom), double buffered.  Every sum runs in a fixed order:
// deterministic.
#include <hip/hip_runtime.h>

#include "gemm_core.hpp"
#include "index_math.hpp"
#include "launch_conv.hpp"

namespace ntk {

constexpr int kPairDMax = 64;   // image pixels the pair kernel takes (PK held in registers)

// G [M*O, D, C] -> Gt [M, C, O, Dp]: for every sample and channel the O x D cotangent block,
// its pixel rows padded with zeros to Dp.  One workgroup per (cotangent image, 64 channels):
// the D x 64 block is read along c, transposed through LDS and written along p.
__global__ void __launch_bounds__(256)
k_pair_gt(const float* __restrict__ G, int O, int D, int C, int Dp, float* __restrict__ Gt) {
  __shared__ float t[64][kPairDMax + 1];
  const int mo = blockIdx.x;                 // cotangent image m * O + o
  const int c0 = blockIdx.y * 64;
  const int m = mo / O, o = mo - m * O;
  const float* src = G + (long long)mo * D * C;
  for (int q = threadIdx.x; q < Dp * 64; q += 256) {
    const int p = q >> 6, c = q & 63;
    t[c][p] = (p < D && c0 + c < C) ? src[(long long)p * C + c0 + c] : 0.f;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < 64 * Dp; q += 256) {
    const int c = q / Dp, p = q - c * Dp;
    if (c0 + c < C) Gt[(((long long)m * C + c0 + c) * O + o) * Dp + p] = t[c][p];
  }
}

struct PairMfmaArgs {
  const float* h;      // layer input of the stacked batch [M, D, Cin]
  const float* Gt;     // its output cotangent, laid out [M, C, O, Dp]
  const float* gram;   // readout summand: [n1, n2] (g1 . g2), or [n] on the batch diagonal
  float* theta;
  int n1, n2, n2_off, O, H, W, D, Cin, C, taps;
  int nob;             // output blocks of 16 along o: ceil(O / 16)
  int nb2;             // pair blocks along batch 2
  int nblk;            // pair blocks
  int accumulate, trace;
  int vec4;            // the layer input rows can be read as float4 (Cin % 4 == 0, aligned)
};

// Geometry of one instantiation, DT blocks of 16 pixels:
//  * pairs per wave PPW: two for images of at most 16 pixels (one sample of batch 1 against two
//    of batch 2: the G1 operand of a channel is read once for the two; with four pairs per wave
//    the 4x4-image CNN's 64 x 64 pairs leave one wave per SIMD, 196 vs 177 us for three layers,
//    and one pair per wave took 203), one otherwise (the PK registers of more would not fit);
//  * a workgroup of 4 waves takes B1 x B2 input pairs (4 x PPW, or 2 x 2), or with DIAG four pairs
//    (n, n) of the batch diagonal; its NS = B1 + B2 sample slots (batch 1, then batch 2) are staged
//    per chunk of CC channels, 16 cotangent rows x Dp pixels per slot and channel, each row padded
//    by 4 floats so that the 16 rows one 16-byte read touches fall in 16 distinct bank groups.
constexpr int kPairsPerWave16 = 2;   // pairs per wave for images of at most 16 pixels

template <int DT, bool DIAG>
struct PairGeom {
  static constexpr int Dp = 16 * DT;
  static constexpr int LD = Dp + 4;
  static constexpr int PPW = (DT == 1 && !DIAG) ? kPairsPerWave16 : 1;
  static constexpr int B1 = DIAG ? 4 : (PPW > 1 ? 4 : 2);
  static constexpr int B2 = DIAG ? 4 : (PPW > 1 ? PPW : 2);
  static constexpr int NS = B1 + B2;
  static constexpr int CC0 = 512 / (NS * LD);             // two chunks in about 64 KB of LDS
  static constexpr int CC = CC0 > 0 ? CC0 : 1;
  static constexpr int ROWS = NS * CC * 16;
  static constexpr int CHUNK = ROWS * LD;                 // floats of one chunk buffer
  static constexpr int NU = ROWS * Dp / 4 / 256;          // float4 loads per thread per chunk
  static_assert(ROWS * Dp / 4 % 256 == 0, "a chunk splits evenly into float4 loads");
  // the pixel Grams of every wave's pairs, rows LD = Dp + 4 floats apart: the four lane groups
  // of a PK read (rows 4g + j) then fall 16 banks apart
  static constexpr int HFLOATS = 4 * PPW * Dp * LD;
  static constexpr int SMEM = (2 * CHUNK > HFLOATS ? 2 * CHUNK : HFLOATS) * 4;
};

__device__ __forceinline__ float wave_sum64(float v) {
  // butterfly over the 64 lanes (DPP within rows, then across rows), fixed order
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xA, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xC, 0xF, false));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Two workgroups fit a compute unit's LDS, so up to 256 registers per lane are free to use.
template <int DT, bool DIAG>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 2)))
k_pairsum_mfma(PairMfmaArgs a) {
  using Gm = PairGeom<DT, DIAG>;
  constexpr int Dp = Gm::Dp, LD = Gm::LD, NS = Gm::NS, CC = Gm::CC, NU = Gm::NU, PPW = Gm::PPW;
  constexpr int B1 = Gm::B1, B2 = Gm::B2;
  extern __shared__ float sm[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, li = lane & 15;
  int blk;
  if (!xcd_block(blockIdx.x, a.nblk, blk)) return;
  const int D = a.D, O = a.O, C = a.C;

  // sample slots (rows of the stacked batch) and this wave's pairs: slot s1 of batch 1 against the
  // slots s2[p] of batch 2, pair indices (i1, i2[p])
  int slot_m[NS];
  bool slot_ok[NS];
  int i1, i2[PPW], s1, s2[PPW];
  if constexpr (DIAG) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int n = 4 * blk + k;
      slot_ok[k] = slot_ok[4 + k] = n < a.n1;
      slot_m[k] = min(n, a.n1 - 1);
      slot_m[4 + k] = a.n2_off + slot_m[k];
    }
    i1 = i2[0] = 4 * blk + wave;
    s1 = wave;
    s2[0] = 4 + wave;
  } else {
    const int bi = blk / a.nb2, bj = blk - bi * a.nb2;
#pragma unroll
    for (int k = 0; k < B1; ++k) {
      slot_ok[k] = B1 * bi + k < a.n1;
      slot_m[k] = min(B1 * bi + k, a.n1 - 1);
    }
#pragma unroll
    for (int k = 0; k < B2; ++k) {
      slot_ok[B1 + k] = B2 * bj + k < a.n2;
      slot_m[B1 + k] = a.n2_off + min(B2 * bj + k, a.n2 - 1);
    }
    if constexpr (PPW > 1) {
      s1 = wave;
      i1 = B1 * bi + wave;
#pragma unroll
      for (int p = 0; p < PPW; ++p) {
        s2[p] = B1 + p;
        i2[p] = B2 * bj + p;
      }
    } else {
      s1 = wave >> 1;
      s2[0] = B1 + (wave & 1);
      i1 = 2 * bi + (wave >> 1);
      i2[0] = 2 * bj + (wave & 1);
    }
  }
  bool active[PPW];
#pragma unroll
  for (int p = 0; p < PPW; ++p) active[p] = DIAG ? i1 < a.n1 : (i1 < a.n1 && i2[p] < a.n2);

  // ---- the staging units of this thread: unit u -> (slot k, channel c, row r, pixel quad p4)
  int u_goff[NU], u_loff[NU], u_c[NU], u_k[NU], u_r[NU];
#pragma unroll
  for (int n = 0; n < NU; ++n) {
    const int u = tid + n * 256;
    const int r = u & 15, rest = u >> 4;
    const int p4 = rest % (Dp / 4), rest2 = rest / (Dp / 4);
    const int c = rest2 % CC, k = rest2 / CC;
    u_r[n] = r;
    u_c[n] = c;
    u_k[n] = k;
    u_loff[n] = ((k * CC + c) * 16 + r) * LD + 4 * p4;
    u_goff[n] = 4 * p4;
  }
  // global offset (without the channel; always a valid address) and validity of each unit for an
  // output block; the loads are unconditional and the zeros are applied at the LDS store
  int base[NU];
  bool uok[NU];
  auto setup_block = [&](int ob1, int ob2) {
#pragma unroll
    for (int n = 0; n < NU; ++n) {
      const int k = u_k[n];
      const int o = (k < B1 ? 16 * ob1 : 16 * ob2) + u_r[n];
      uok[n] = slot_ok[k] && o < O;
      base[n] = (slot_m[k] * C * O + min(o, O - 1)) * Dp + u_goff[n];
    }
  };
  unsigned okm = 0;   // bit n: unit n of the chunk in flight is inside the operand
  auto load_chunk = [&](int c0, f32x4 (&rg)[NU]) {
    okm = 0;
#pragma unroll
    for (int n = 0; n < NU; ++n) {
      const int ch = c0 + u_c[n];
      okm |= (uok[n] && ch < C) ? (1u << n) : 0u;
      rg[n] = *reinterpret_cast<const f32x4*>(a.Gt + base[n] + min(ch, C - 1) * O * Dp);
    }
  };
  auto store_chunk = [&](float* buf, const f32x4 (&rg)[NU]) {
#pragma unroll
    for (int n = 0; n < NU; ++n) {
      const f32x4 z = {0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4*>(buf + u_loff[n]) = (okm >> n) & 1u ? rg[n] : z;
    }
  };
  const int ob_n = a.trace ? a.nob : 1;
  auto block_of = [&](int ob, int& ob1, int& ob2) {
    ob1 = a.trace ? ob : (int)blockIdx.y / a.nob;
    ob2 = a.trace ? ob : (int)blockIdx.y - ob1 * a.nob;
  };
  // the first chunk of cotangents is in flight while the patch-pair Grams are formed
  f32x4 rg[NU];
  {
    int ob1, ob2;
    block_of(0, ob1, ob2);
    setup_block(ob1, ob2);
    load_chunk(0, rg);
  }

  // ---- pixel Grams H of this wave's pairs (16 x 16 blocks, K = Cin), staged in LDS
  {
    const float* h1 = a.h + (long long)slot_m[s1] * D * a.Cin;
    const float* h2[PPW];
#pragma unroll
    for (int p = 0; p < PPW; ++p) h2[p] = a.h + (long long)slot_m[s2[p]] * D * a.Cin;
    f32x4 hc[PPW][DT][DT];
#pragma unroll
    for (int p = 0; p < PPW; ++p)
#pragma unroll
      for (int r = 0; r < DT; ++r)
#pragma unroll
        for (int s = 0; s < DT; ++s) hc[p][r][s] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto gram_step = [&](int k0, const float (&av)[DT][4], const float (&bv)[PPW][DT][4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int p = 0; p < PPW; ++p)
#pragma unroll
          for (int r = 0; r < DT; ++r)
#pragma unroll
            for (int s = 0; s < DT; ++s)
              hc[p][r][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[r][j], bv[p][s][j], hc[p][r][s], 0, 0, 0);
    };
    if (a.vec4) {
      // Cin % 4 == 0 and 16-byte aligned rows: lane (i, g) reads ci = k0 + 4g .. k0 + 4g + 3 of its
      // pixel row at once (zeros past Cin come in whole quads)
#pragma unroll 2
      for (int k0 = 0; k0 < a.Cin; k0 += 16) {
        float av[DT][4], bv[PPW][DT][4];
        const int ci = k0 + 4 * g;
        const bool cok = ci < a.Cin;
        const int cc = min(ci, a.Cin - 4);
#pragma unroll
        for (int r = 0; r < DT; ++r) {
          const int q = 16 * r + li, qc = min(q, D - 1);
          const bool ok = cok && q < D;
          const f32x4 x1 = *reinterpret_cast<const f32x4*>(h1 + (long long)qc * a.Cin + cc);
#pragma unroll
          for (int j = 0; j < 4; ++j) av[r][j] = ok ? x1[j] : 0.f;
#pragma unroll
          for (int p = 0; p < PPW; ++p) {
            const f32x4 x2 = *reinterpret_cast<const f32x4*>(h2[p] + (long long)qc * a.Cin + cc);
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[p][r][j] = ok ? x2[j] : 0.f;
          }
        }
        gram_step(k0, av, bv);
      }
    } else {
      for (int k0 = 0; k0 < a.Cin; k0 += 16) {
        float av[DT][4], bv[PPW][DT][4];
#pragma unroll
        for (int r = 0; r < DT; ++r) {
          const int q = 16 * r + li, qc = min(q, D - 1);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int ci = k0 + 4 * g + j, cc = min(ci, a.Cin - 1);
            const bool ok = q < D && ci < a.Cin;
            const float x1 = h1[(long long)qc * a.Cin + cc];
            av[r][j] = ok ? x1 : 0.f;
#pragma unroll
            for (int p = 0; p < PPW; ++p) {
              const float x2 = h2[p][(long long)qc * a.Cin + cc];
              bv[p][r][j] = ok ? x2 : 0.f;
            }
          }
        }
        gram_step(k0, av, bv);
      }
    }
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      float* Hs = sm + (wave * PPW + p) * Dp * LD;
#pragma unroll
      for (int r = 0; r < DT; ++r)
#pragma unroll
        for (int s = 0; s < DT; ++s)
#pragma unroll
          for (int v = 0; v < 4; ++v) Hs[(16 * r + 4 * g + v) * LD + 16 * s + li] = hc[p][r][s][v];
    }
  }
  __syncthreads();
  float pk[PPW][DT][DT][4];
  // ---- this lane's PK entries (the A operands of the X products).  Both patches of a PK entry
  // take the same tap, so tap (dy, dx) adds H[p1 + s, p2 + s] with s = dy W + dx, i.e. the entry
  // (dy W + dx)(LD + 1) further on, when both shifted pixels lie inside the image: a 9-bit mask
  // per pixel (bit 3 (dy + 1) + dx + 1), formed once per pixel the lane touches.
  auto tapmask = [&](int p) -> unsigned {
    if (p >= D) return 0u;
    const int y = p / a.W, x = p - y * a.W;
    unsigned m = 0;
#pragma unroll
    for (int dy = -1; dy <= 1; ++dy)
#pragma unroll
      for (int dx = -1; dx <= 1; ++dx)
        if ((unsigned)(y + dy) < (unsigned)a.H && (unsigned)(x + dx) < (unsigned)a.W) m |= 1u << (3 * (dy + 1) + dx + 1);
    return m;
  };
  unsigned m1[DT][4], m2[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) {
    m2[t] = tapmask(16 * t + li);
#pragma unroll
    for (int j = 0; j < 4; ++j) m1[t][j] = tapmask(16 * t + 4 * g + j);
  }
  const int W = a.W;
#pragma unroll
  for (int p = 0; p < PPW; ++p) {
    const float* Hs = sm + (wave * PPW + p) * Dp * LD;
#pragma unroll
    for (int rt = 0; rt < DT; ++rt)
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const unsigned m = m1[t][j] & m2[rt];
          const int e = (16 * t + 4 * g + j) * LD + 16 * rt + li;   // H[p1][p2]
          float v;
          if (a.taps == 1) {
            v = (m >> 4) & 1u ? Hs[e] : 0.f;
          } else {
            v = 0.f;
#pragma unroll
            for (int dy = -1; dy <= 1; ++dy)
#pragma unroll
              for (int dx = -1; dx <= 1; ++dx) {
                const int k = 3 * (dy + 1) + dx + 1;
                // a masked tap reads a clamped, valid address and adds nothing
                const int ee = min(max(e + (dy * W + dx) * (LD + 1), 0), Dp * LD - 1);
                const float hv = Hs[ee];
                v += (m >> k) & 1u ? hv : 0.f;
              }
          }
          pk[p][rt][t][j] = v;
        }
  }
  __syncthreads();   // the pixel Grams' LDS is reused by the cotangent chunks

  float tr[PPW];
#pragma unroll
  for (int p = 0; p < PPW; ++p) tr[p] = 0.f;
  for (int ob = 0; ob < ob_n; ++ob) {
    int ob1, ob2;
    block_of(ob, ob1, ob2);
    if (ob > 0) {
      setup_block(ob1, ob2);
      load_chunk(0, rg);
    }
    f32x4 acc[PPW][2];
#pragma unroll
    for (int p = 0; p < PPW; ++p) acc[p][0] = acc[p][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    store_chunk(sm, rg);
    __syncthreads();
    const int nchunk = (C + CC - 1) / CC;   // the channels past C of the last chunk hold zeros
    for (int q = 0; q < nchunk; ++q) {
      const float* buf = sm + (q & 1) * Gm::CHUNK;
      if (q + 1 < nchunk) load_chunk((q + 1) * CC, rg);
      // every B operand of the chunk first (one 16-byte LDS read per 16 pixels, channel and
      // slot), so that the reads are in flight together
      f32x4 b1[CC][DT], b2[CC][PPW][DT];
#pragma unroll
      for (int c = 0; c < CC; ++c)
#pragma unroll
        for (int t = 0; t < DT; ++t) {
          b1[c][t] = *reinterpret_cast<const f32x4*>(buf + ((s1 * CC + c) * 16 + li) * LD + 16 * t + 4 * g);
#pragma unroll
          for (int p = 0; p < PPW; ++p)
            b2[c][p][t] = *reinterpret_cast<const f32x4*>(buf + ((s2[p] * CC + c) * 16 + li) * LD + 16 * t + 4 * g);
        }
      // X^T of every pair for channel c (DT blocks of 16 pixels p2), from the PK registers and G1
      auto xprod = [&](int c, f32x4 (&X)[PPW][DT]) {
#pragma unroll
        for (int p = 0; p < PPW; ++p)
#pragma unroll
          for (int rt = 0; rt < DT; ++rt) {
            X[p][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
              for (int j = 0; j < 4; ++j)
                X[p][rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(pk[p][rt][t][j], b1[c][t][j], X[p][rt], 0, 0, 0);
          }
      };
      // theta += X G2 of every pair for channel c
      auto tprod = [&](int c, const f32x4 (&X)[PPW][DT]) {
#pragma unroll
        for (int p = 0; p < PPW; ++p)
#pragma unroll
          for (int rt = 0; rt < DT; ++rt)
#pragma unroll
            for (int v = 0; v < 4; ++v)
              acc[p][c & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(X[p][rt][v], b2[c][p][rt][v], acc[p][c & 1], 0, 0, 0);
      };
      // software pipeline over the chunk's channels: the X products of channel c + 1 issue before
      // the theta products of channel c (pairs past the batch compute on clamped samples and
      // write nothing)
      f32x4 Xa[PPW][DT], Xb[PPW][DT];
      xprod(0, Xa);
#pragma unroll
      for (int c = 0; c < CC; ++c) {
        if (c + 1 < CC) {
          if (c & 1) xprod(c + 1, Xa); else xprod(c + 1, Xb);
        }
        if (c & 1) tprod(c, Xb); else tprod(c, Xa);
      }
      if (q + 1 < nchunk) {
        store_chunk(sm + ((q + 1) & 1) * Gm::CHUNK, rg);
        __syncthreads();
      }
    }
    __syncthreads();   // the chunk buffers are refilled by the next output block
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      const f32x4 sum = acc[p][0] + acc[p][1];
      if (a.trace) {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (4 * g + v == li && 16 * ob + li < O) tr[p] += sum[v];
      } else if (active[p]) {
        const long long pair = DIAG ? i1 : (long long)i1 * a.n2 + i2[p];
        const float gr = a.gram[pair];
        float* dst = a.theta + pair * O * O;
        const int o2 = 16 * ob2 + li;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int o1 = 16 * ob1 + 4 * g + v;
          if (o1 < O && o2 < O) {
            float val = sum[v];
            if (a.accumulate)
              val += dst[o1 * O + o2];
            else if (o1 == o2)
              val += gr;
            dst[o1 * O + o2] = val;
          }
        }
      }
    }
  }
  if (a.trace) {
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      const float t = wave_sum64(tr[p]);
      if (active[p] && lane == 0) {
        const long long pair = DIAG ? i1 : (long long)i1 * a.n2 + i2[p];
        float* dst = a.theta + pair;
        *dst = a.accumulate ? *dst + t : t + (float)O * a.gram[pair];
      }
    }
  }
}

int pairsum_supported(int D) { return D >= 1 && D <= kPairDMax; }

long long pairsum_gt_floats(long long images, int O, int D, int C) {
  const int Dp = 16 * ((D + 15) / 16);
  return images * C * O * Dp;
}

template <int DT, bool DIAG>
static hipError_t pairsum_go(hipStream_t s, PairMfmaArgs a, int gy) {
  using Gm = PairGeom<DT, DIAG>;
  long long nblk;
  if (DIAG) {
    nblk = (a.n1 + 3) / 4;
    a.nb2 = 0;
  } else {
    a.nb2 = (a.n2 + Gm::B2 - 1) / Gm::B2;
    nblk = (long long)((a.n1 + Gm::B1 - 1) / Gm::B1) * a.nb2;
  }
  if (nblk >= (1LL << 28)) return hipErrorInvalidValue;
  a.nblk = (int)nblk;
  hipError_t e = hipFuncSetAttribute((const void*)k_pairsum_mfma<DT, DIAG>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, Gm::SMEM);
  if (e != hipSuccess) return e;
  const int grid = 8 * ((a.nblk + 7) / 8);
  k_pairsum_mfma<DT, DIAG><<<dim3(grid, gy), dim3(256), Gm::SMEM, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_conv_pairsum(hipStream_t s, const float* h, const float* G, float* Gt, int n1, int n2,
                               int n2_offset, int O, int H, int W, int Cin, int C, int taps,
                               const float* gram, int accumulate, int trace, int diag, float* theta) {
  const int D = H * W;
  if (!pairsum_supported(D) || (diag && n1 != n2) || (taps != 1 && taps != 9)) return hipErrorInvalidValue;
  const int DT = (D + 15) / 16, Dp = 16 * DT;
  const int images = n2_offset + n2 > n1 ? n2_offset + n2 : n1;   // rows of the stacked batch in use
  {
    const long long blocks = (long long)images * O;
    if (blocks >= (1LL << 31)) return hipErrorInvalidValue;
    k_pair_gt<<<dim3((unsigned)blocks, (C + 63) / 64), dim3(256), 0, s>>>(G, O, D, C, Dp, Gt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  PairMfmaArgs a{};
  a.h = h;
  a.Gt = Gt;
  a.gram = gram;
  a.theta = theta;
  a.n1 = n1;
  a.n2 = n2;
  a.n2_off = n2_offset;
  a.O = O;
  a.H = H;
  a.W = W;
  a.D = D;
  a.Cin = Cin;
  a.C = C;
  a.taps = taps;
  a.nob = (O + 15) / 16;
  a.accumulate = accumulate;
  a.trace = trace;
  a.vec4 = Cin % 4 == 0 && (reinterpret_cast<uintptr_t>(h) & 15) == 0;
  const int gy = trace ? 1 : a.nob * a.nob;
  if (gy > 65535) return hipErrorInvalidValue;
  switch (DT) {
    case 1: return diag ? pairsum_go<1, true>(s, a, gy) : pairsum_go<1, false>(s, a, gy);
    case 2: return diag ? pairsum_go<2, true>(s, a, gy) : pairsum_go<2, false>(s, a, gy);
    case 3: return diag ? pairsum_go<3, true>(s, a, gy) : pairsum_go<3, false>(s, a, gy);
    default: return diag ? pairsum_go<4, true>(s, a, gy) : pairsum_go<4, false>(s, a, gy);
  }
}

}  // namespace ntk
