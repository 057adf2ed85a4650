// gemm_core.hpp -- fp32 MFMA building blocks for gfx950 (CDNA4).
//
// Every contraction of the structured-derivatives NTK is a dense fp32 product
// C[M,N] = sum_k A[m,k] B[n,k] with operands that are either K-contiguous in
// memory ("K-inner": a row of K values is contiguous) or row-contiguous
// ("K-outer": for a fixed k the rows are contiguous).  The blocks below stage
// BM x BK and BN x BK tiles through LDS (double buffered, one barrier per K
// tile) and run v_mfma_f32_32x32x2_f32 on 32x32 fragments held by each wave.
//
// MFMA 32x32x2 f32 operand layout (lane l of a 64-wide wave):
//   A: lane l supplies A[i = l % 32][k = l / 32]
//   B: lane l supplies B[k = l / 32][j = l % 32]
//   D: lane l, register v holds D[i = 8*(v/4) + 4*(l/32) + (v%4)][j = l % 32]
// A K-step of 8 is split as k = kk + 4*(l/32) + t for the t-th of four MFMAs, so
// each lane fetches 4 consecutive k of its row with one 16-byte LDS read when the
// LDS tile is K-inner.  The summation over k is order free, and A and B use the
// same k assignment, so the product is the plain sum over the 8 k values.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "index_math.hpp"

namespace ntk {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------------------ tile config
template <int BM_, int BN_, int BK_, int WM_, int WN_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
  static constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
  static constexpr int WAVES = WAVES_M * WAVES_N;
  static constexpr int THREADS = WAVES * 64;
  static constexpr int FM = WM / 32, FN = WN / 32;      // 32x32 fp32 fragments per wave
  static constexpr int FM16 = WM / 16, FN16 = WN / 16;  // 16x16 fp64 fragments per wave
  static_assert(BM % WM == 0 && BN % WN == 0, "wave tiling");
  static_assert(WM % 16 == 0 && WN % 16 == 0, "MFMA fragments");
  static_assert(BK % 16 == 0, "K tile is a multiple of 16");
};

// LDS tile geometry.  K-inner: [ROWS][BK + 4] (16-byte reads of 4 k per lane hit 16
// distinct bank groups for 16 consecutive rows).  K-outer: [BK][ROWS + 8] (lanes 0-31
// and 32-63 read rows k and k+4, 4*(ROWS+8) = 32 mod 64 banks apart).
template <int ROWS, int BK, bool K_INNER>
struct LdsGeom {
  static constexpr int LD = K_INNER ? (BK + 4) : (ROWS + 8);
  static constexpr int FLOATS = K_INNER ? ROWS * LD : BK * LD;
};

// ------------------------------------------------------------------------------ global -> regs -> LDS
// A loader provides
//   static constexpr bool K_INNER;
//   __device__ f32x4 load4(int row, int k, uint32_t& valid) const;
// returning the raw elements (row, k..k+3) if K_INNER, else (row..row+3, k), read from
// clamped in-range addresses, with bit j of `valid` set when element j is inside the
// operand.  The zero fill of invalid elements happens at the LDS store, so the selects do
// not wait on the global loads and the prefetch stays in flight across the MFMA stage.
//
// A loader may also keep per-row state: it then defines
//   struct RowState;  __device__ RowState row_state(int row) const;
//   __device__ f32x4 load4s(const RowState&, int k, uint32_t& valid) const;
// and TileIO computes the state of each of its rows once per tile (prepare), so the index
// arithmetic that depends only on the row (image, pixel, channel block, ...) leaves the K loop.
template <class L, class = void>
struct has_row_state : std::false_type {};
template <class L>
struct has_row_state<L, std::void_t<typename L::RowState>> : std::true_type {};
// A loader whose 4 elements are always valid together (all or none) sets
//   static constexpr bool UNIFORM_VALID = true;
// and the LDS store then tests one condition instead of four bits.
template <class L, class = void>
struct uniform_valid : std::false_type {};
template <class L>
struct uniform_valid<L, std::void_t<decltype(L::UNIFORM_VALID)>> : std::integral_constant<bool, L::UNIFORM_VALID> {};

template <class L, bool = has_row_state<L>::value>
struct row_state_of {
  using type = int;
};
template <class L>
struct row_state_of<L, true> {
  using type = typename L::RowState;
};

template <class Loader, int ROWS, int BK, int THREADS>
struct TileIO {
  static constexpr bool KI = Loader::K_INNER;
  static constexpr bool RS = has_row_state<Loader>::value;
  static constexpr int NV = ROWS * BK / (4 * THREADS);
  static_assert(ROWS * BK % (4 * THREADS) == 0, "tile must split evenly into float4 per thread");
  using G = LdsGeom<ROWS, BK, KI>;
  using State = typename row_state_of<Loader>::type;
  f32x4 r[NV];
  uint32_t m[NV];
  State st[NV];

  // row and k offset of this thread's i-th float4 of the tile
  __device__ __forceinline__ static int slot_row(int q) {
    return KI ? q / (BK / 4) : (q % (ROWS / 4)) * 4;
  }
  __device__ __forceinline__ static int slot_k(int q) {
    return KI ? (q % (BK / 4)) * 4 : q / (ROWS / 4);
  }
  __device__ __forceinline__ void prepare(const Loader& ld, int row0, int tid) {
    if constexpr (RS) {
#pragma unroll
      for (int i = 0; i < NV; ++i) st[i] = ld.row_state(row0 + slot_row(tid + i * THREADS));
    }
  }
  __device__ __forceinline__ void load(const Loader& ld, int row0, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int q = tid + i * THREADS;
      if constexpr (RS)
        r[i] = ld.load4s(st[i], k0 + slot_k(q), m[i]);
      else
        r[i] = ld.load4(row0 + slot_row(q), k0 + slot_k(q), m[i]);
    }
  }
  __device__ __forceinline__ void store(float* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int q = tid + i * THREADS;
      f32x4 v = r[i];
      if constexpr (uniform_valid<Loader>::value) {
        const bool ok = m[i] != 0u;
        v[0] = ok ? v[0] : 0.f;
        v[1] = ok ? v[1] : 0.f;
        v[2] = ok ? v[2] : 0.f;
        v[3] = ok ? v[3] : 0.f;
      } else {
        v[0] = (m[i] & 1u) ? v[0] : 0.f;
        v[1] = (m[i] & 2u) ? v[1] : 0.f;
        v[2] = (m[i] & 4u) ? v[2] : 0.f;
        v[3] = (m[i] & 8u) ? v[3] : 0.f;
      }
      if (KI)
        *reinterpret_cast<f32x4*>(&lds[slot_row(q) * G::LD + slot_k(q)]) = v;
      else
        *reinterpret_cast<f32x4*>(&lds[slot_k(q) * G::LD + slot_row(q)]) = v;
    }
  }
};

// 4 consecutive k of one row from an LDS tile.
template <bool KI, int LD>
__device__ __forceinline__ f32x4 frag_read(const float* lds, int row, int k) {
  if (KI) {
    return *reinterpret_cast<const f32x4*>(&lds[row * LD + k]);
  } else {
    f32x4 v;
    v[0] = lds[(k + 0) * LD + row];
    v[1] = lds[(k + 1) * LD + row];
    v[2] = lds[(k + 2) * LD + row];
    v[3] = lds[(k + 3) * LD + row];
    return v;
  }
}

// One LDS stage: acc[fm][fn] += A_tile(wave rows) * B_tile(wave cols)^T over BK.  The
// fragments of K step kk+8 are read while the MFMAs of step kk issue (two fragment
// buffers), and a scheduling fence per step keeps the compiler from hoisting every
// fragment read of the stage (which would cost 4x the fragment registers).
template <class Cfg, bool AKI, bool BKI>
__device__ __forceinline__ void mma_stage(const float* As, const float* Bs,
                                          f32x16 (&acc)[Cfg::FM][Cfg::FN], int wm0, int wn0,
                                          int lane) {
  using GA = LdsGeom<Cfg::BM, Cfg::BK, AKI>;
  using GB = LdsGeom<Cfg::BN, Cfg::BK, BKI>;
  const int lr = lane & 31, lk = (lane >> 5) * 4;
  f32x4 a[2][Cfg::FM], b[2][Cfg::FN];
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm) a[0][fm] = frag_read<AKI, GA::LD>(As, wm0 + fm * 32 + lr, lk);
#pragma unroll
  for (int fn = 0; fn < Cfg::FN; ++fn) b[0][fn] = frag_read<BKI, GB::LD>(Bs, wn0 + fn * 32 + lr, lk);
#pragma unroll
  for (int kk = 0; kk < Cfg::BK; kk += 8) {
    const int cur = (kk / 8) & 1;
    if (kk + 8 < Cfg::BK) {
#pragma unroll
      for (int fm = 0; fm < Cfg::FM; ++fm)
        a[cur ^ 1][fm] = frag_read<AKI, GA::LD>(As, wm0 + fm * 32 + lr, kk + 8 + lk);
#pragma unroll
      for (int fn = 0; fn < Cfg::FN; ++fn)
        b[cur ^ 1][fn] = frag_read<BKI, GB::LD>(Bs, wn0 + fn * 32 + lr, kk + 8 + lk);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < Cfg::FN; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[cur][fm][t], b[cur][fn][t], acc[fm][fn], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <class Cfg>
__device__ __forceinline__ void zero_acc(f32x16 (&acc)[Cfg::FM][Cfg::FN]) {
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[fm][fn][v] = 0.0f;
}

// fp64-accumulated variant for the forward pass: the fp32 LDS fragments are widened
// exactly to fp64 and multiplied with v_mfma_f64_16x16x4_f64, so a pre-activation is
// the fp64 sum of exact products of fp32 inputs (its sign, the ReLU decision, is then
// a deterministic function of the fp32 data).
// MFMA 16x16x4 f64 layout: A: lane l supplies A[i = l % 16][k = l / 16];
//   B: B[k = l / 16][j = l % 16];  D: lane l, element v holds D[4*v + l/16][l % 16]
//   (unlike the fp32 16x16x4 form, the four outputs of a lane are 4 rows apart).
// K step of 16 split as k = kk + 4*(l/16) + t for the t-th of four MFMAs.
template <class Cfg, bool AKI, bool BKI>
__device__ __forceinline__ void mma_stage(const float* As, const float* Bs,
                                          f64x4 (&acc)[Cfg::FM16][Cfg::FN16], int wm0, int wn0,
                                          int lane) {
  using GA = LdsGeom<Cfg::BM, Cfg::BK, AKI>;
  using GB = LdsGeom<Cfg::BN, Cfg::BK, BKI>;
  const int lr = lane & 15, lk = (lane >> 4) * 4;
#pragma unroll
  for (int kk = 0; kk < Cfg::BK; kk += 16) {
    f32x4 a[Cfg::FM16], b[Cfg::FN16];
#pragma unroll
    for (int fm = 0; fm < Cfg::FM16; ++fm) a[fm] = frag_read<AKI, GA::LD>(As, wm0 + fm * 16 + lr, kk + lk);
#pragma unroll
    for (int fn = 0; fn < Cfg::FN16; ++fn) b[fn] = frag_read<BKI, GB::LD>(Bs, wn0 + fn * 16 + lr, kk + lk);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int fm = 0; fm < Cfg::FM16; ++fm)
#pragma unroll
        for (int fn = 0; fn < Cfg::FN16; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a[fm][t], (double)b[fn][t],
                                                             acc[fm][fn], 0, 0, 0);
  }
}

template <class Cfg>
__device__ __forceinline__ void zero_acc(f64x4 (&acc)[Cfg::FM16][Cfg::FN16]) {
#pragma unroll
  for (int fm = 0; fm < Cfg::FM16; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN16; ++fn)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[fm][fn][v] = 0.0;
}

template <class Cfg, class F>
__device__ __forceinline__ void for_each_acc(f64x4 (&acc)[Cfg::FM16][Cfg::FN16], int m0, int n0, F&& f) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
#pragma unroll
  for (int fm = 0; fm < Cfg::FM16; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN16; ++fn)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = m0 + wm0 + fm * 16 + 4 * v + (lane >> 4);
        const int col = n0 + wn0 + fn * 16 + (lane & 15);
        f(row, col, acc[fm][fn][v]);
      }
}

// Full K loop over [k_begin, k_end) for the tile (m0, n0): double-buffered LDS, one
// barrier per K tile.  `smem` holds 2 * (A tile + B tile) floats.  Ends with a barrier,
// so the caller may reuse `smem` afterwards.  AccT selects the MFMA flavour (fp32
// 32x32x2 fragments or fp64 16x16x4 fragments).
template <class Cfg, class LA, class LB, class AccT>
__device__ __forceinline__ void gemm_mainloop(const LA& la, const LB& lb, int m0, int n0, int k_begin,
                                              int k_end, float* smem, AccT& acc) {
  using GA = LdsGeom<Cfg::BM, Cfg::BK, LA::K_INNER>;
  using GB = LdsGeom<Cfg::BN, Cfg::BK, LB::K_INNER>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
  // stage s of the double buffer: A at smem + s * STAGE, B right after it.  Offsets (not an
  // array of pointers) keep every access in the LDS address space (ds_read / ds_write).
  constexpr int STAGE = GA::FLOATS + GB::FLOATS;

  const int nk = (k_end - k_begin + Cfg::BK - 1) / Cfg::BK;
  if (nk <= 0) return;
  TileIO<LA, Cfg::BM, Cfg::BK, Cfg::THREADS> ia;
  TileIO<LB, Cfg::BN, Cfg::BK, Cfg::THREADS> ib;
  ia.prepare(la, m0, tid);
  ib.prepare(lb, n0, tid);
  ia.load(la, m0, k_begin, tid);
  ib.load(lb, n0, k_begin, tid);
  ia.store(smem, tid);
  ib.store(smem + GA::FLOATS, tid);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = (kt & 1) * STAGE, nxt = STAGE - cur;
    const bool more = kt + 1 < nk;
    if (more) {
      ia.load(la, m0, k_begin + (kt + 1) * Cfg::BK, tid);
      ib.load(lb, n0, k_begin + (kt + 1) * Cfg::BK, tid);
    }
    mma_stage<Cfg, LA::K_INNER, LB::K_INNER>(smem + cur, smem + cur + GA::FLOATS, acc, wm0, wn0, lane);
    if (more) {
      ia.store(smem + nxt, tid);
      ib.store(smem + nxt + GA::FLOATS, tid);
    }
    __syncthreads();
  }
}

template <class Cfg, class LA, class LB>
constexpr int gemm_smem_bytes() {
  return 2 * (LdsGeom<Cfg::BM, Cfg::BK, LA::K_INNER>::FLOATS +
              LdsGeom<Cfg::BN, Cfg::BK, LB::K_INNER>::FLOATS) * 4;
}

// Visit every accumulator element of the wave with its global (row, col).
template <class Cfg, class F>
__device__ __forceinline__ void for_each_acc(f32x16 (&acc)[Cfg::FM][Cfg::FN], int m0, int n0, F&& f) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm0 + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const int col = n0 + wn0 + fn * 32 + (lane & 31);
        f(row, col, acc[fm][fn][v]);
      }
}

// Two-phase epilogues: first gather one auxiliary value per accumulator element (all loads
// issued before any is used), then combine and store.
template <class Cfg, class L>
__device__ __forceinline__ void gather_acc(float (&g)[Cfg::FM][Cfg::FN][16], int m0, int n0, L&& load) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm0 + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const int col = n0 + wn0 + fn * 32 + (lane & 31);
        g[fm][fn][v] = load(row, col);
      }
}

template <class Cfg, class F>
__device__ __forceinline__ void for_each_acc_aux(f32x16 (&acc)[Cfg::FM][Cfg::FN],
                                                 const float (&g)[Cfg::FM][Cfg::FN][16], int m0, int n0,
                                                 F&& f) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm0 + fm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const int col = n0 + wn0 + fn * 32 + (lane & 31);
        f(row, col, acc[fm][fn][v], g[fm][fn][v]);
      }
}

// Element at a 32-bit byte offset from a base pointer.  With a wave-uniform base this is the
// scalar-base + 32-bit vector-offset addressing form, one instruction per access with no
// 64-bit address arithmetic.  The caller keeps `bytes` below 4 GiB.
__device__ __forceinline__ float& at_bytes(float* base, uint32_t bytes) {
  return *reinterpret_cast<float*>(reinterpret_cast<char*>(base) + bytes);
}
__device__ __forceinline__ const float& at_bytes(const float* base, uint32_t bytes) {
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(base) + bytes);
}

// Row arithmetic of the epilogues below, per 32-row MFMA fragment: lane l holds rows
// r0 + 8*(v/4) + 4*(l/32) + v%4 (v = 0..15) of column l%32 of the fragment.
__device__ __forceinline__ int frag_row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }

// Epilogue of the cotangent backward through a convolution (3x3 or pointwise):
// out[r, c] = acc[r, c] * dphi[img*D + p, c] for rows r = (img*O + o)*D + p of the O cotangent
// images of each image (null dphi: the identity).  A fragment that lies inside R and inside
// one cotangent image (no multiple of D in (r0, r0 + 31]) maps to 32 consecutive rows of dphi,
// so its row arithmetic is done once and an element costs an offset, a load, a multiply and a
// store (32-bit byte offsets: N < 2^25); other fragments take the per-element form.
template <class Cfg>
__device__ __forceinline__ void store_pixel_rows(f32x16 (&acc)[Cfg::FM][Cfg::FN], int m0, int n0,
                                                 const float* __restrict__ dphi, float* __restrict__ out, int R,
                                                 int N, FastDiv fOD, FastDiv fD) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
  const int D = (int)fD.d;
#pragma unroll
  for (int fm = 0; fm < Cfg::FM; ++fm) {
    const int r0 = __builtin_amdgcn_readfirstlane(m0 + wm0 + fm * 32);
    if (r0 >= R) continue;
    const int t0 = (int)fD.div(r0);
    if (r0 + 32 <= R && N < (1 << 25) && (int)fD.div(r0 + 31) == t0) {
      const int img = (int)fOD.div(r0);
      float* ob = out + (long long)r0 * N;
      const float* db = dphi ? dphi + ((long long)img * D + (r0 - t0 * D)) * N : nullptr;
#pragma unroll
      for (int fn = 0; fn < Cfg::FN; ++fn) {
        const int c = n0 + wn0 + fn * 32 + (lane & 31);
        if (c >= N) continue;
        if (db) {
          float d[16];
#pragma unroll
          for (int v = 0; v < 16; ++v) d[v] = at_bytes(db, (uint32_t)(frag_row(v, lane) * N + c) * 4u);
#pragma unroll
          for (int v = 0; v < 16; ++v) at_bytes(ob, (uint32_t)(frag_row(v, lane) * N + c) * 4u) = acc[fm][fn][v] * d[v];
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) at_bytes(ob, (uint32_t)(frag_row(v, lane) * N + c) * 4u) = acc[fm][fn][v];
        }
      }
    } else {
#pragma unroll
      for (int fn = 0; fn < Cfg::FN; ++fn)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = r0 + frag_row(v, lane), c = n0 + wn0 + fn * 32 + (lane & 31);
          if (r < R && c < N) {
            const int img = (int)fOD.div(r);
            const int p = r - (int)fD.div(r) * D;
            const float d = dphi ? dphi[((long long)img * D + p) * N + c] : 1.f;
            out[(long long)r * N + c] = acc[fm][fn][v] * d;
          }
        }
    }
  }
}

// ------------------------------------------------------------------------------ loaders
// Loaders never branch: an out-of-range element is read from a clamped (valid) address and
// replaced by 0 with a select, so the main loop has no divergent control flow.
//
// Row-major [rows, K] operand with row stride `ld` (floats), K contiguous.  VEC = whole
// float4 loads: requires p 16-byte aligned, ld % 4 == 0 and K % 4 == 0.
template <bool VEC>
struct LoadKInnerT {
  static constexpr bool K_INNER = true;
  static constexpr bool UNIFORM_VALID = VEC;   // VEC: the 4 elements are valid together
  const float* p;
  int rows, K;
  long long ld;
  __device__ __forceinline__ f32x4 load4(int row, int k, uint32_t& valid) const {
    const int rc = min(row, rows - 1);
    if (VEC) {
      const int kc = min(k, K - 4);
      valid = (row < rows && k < K) ? 0xFu : 0u;
      return *reinterpret_cast<const f32x4*>(p + (long long)rc * ld + kc);
    } else {
      f32x4 v;
      valid = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kc = min(k + j, K - 1);
        v[j] = p[(long long)rc * ld + kc];
        valid |= (row < rows && k + j < K) ? (1u << j) : 0u;
      }
      return v;
    }
  }
};
using LoadKInner = LoadKInnerT<true>;

// The VEC form is usable when every pointer is 16-byte aligned and the strides and K are
// multiples of 4 floats.
__host__ inline bool vec_ok(const void* p, long long ld, long long K) {
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 4 == 0 && K % 4 == 0;
}

// ------------------------------------------------------------------------------ misc
__device__ __forceinline__ float act_fwd(int act, float z) {
  if (act == 1) return z > 0.f ? z : 0.f;
  if (act == 2) return erff(z);
  return z;
}
// derivative of the activation at z: ReLU'(0) = 0, erf'(z) = 2/sqrt(pi) exp(-z^2)
__device__ __forceinline__ float act_deriv(int act, float z) {
  if (act == 1) return z > 0.f ? 1.f : 0.f;
  if (act == 2) return 1.1283791670955126f * expf(-z * z);
  return 1.f;
}

}  // namespace ntk

namespace ntk {


}  // namespace ntk

namespace ntk {

// ------------------------------------------------------------------------------ direct-to-LDS main loop
// gfx950 loads global memory straight into LDS (buffer_load_dwordx4 ... lds): lane l of a
// wave writes its 16 bytes at M0 + 16 l, so one instruction fills 1 KB of LDS with no register
// staging and no ds_write.  Tiles are stored unpadded, [rows][BK] with BK = 32 (8 chunks of
// 16 bytes per row), and the chunk c of row r sits at position c ^ ((r >> 1) & 7): the 16
// rows read by a ds_read_b128 then hit 16 distinct 16-byte bank groups.  Two or three LDS
// stages: the next tiles are in flight while tile kt is multiplied, one barrier per K tile.
//
// The row-major operands load through a buffer resource (MUBUF) rather than global_load_lds:
// with a FLAT-encoded LDS load in flight the compiler makes every use of an LDS read wait for
// all LDS reads of the wave, which defeats the fragment prefetch of the main loop.
//
// Requirements (checked by the host): both operands K-contiguous with 16-byte aligned rows
// (LoadKInnerT<true> conditions), K % 32 == 0, and a tile's rows spanning less than 2 GiB.
// Rows past the operand are read from the last row (clamped): they only feed output
// rows/columns that are discarded.
constexpr int kDmaStages = 3;

template <int ROWS>
struct DmaTile {
  static constexpr int BK = 32;
  static constexpr int FLOATS = ROWS * BK;
  __device__ static __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }
  __device__ static __forceinline__ f32x4 frag(const float* lds, int row, int k) {
    return *reinterpret_cast<const f32x4*>(&lds[row * BK + (swz(row, k >> 2) << 2)]);
  }
};

// K-outer form of the tile, for operands whose global memory holds 4 consecutive rows at one
// k (16 bytes): stored [BK][ROWS] (k-major), unpadded.  The 16-byte chunk c of k-row k sits at
// position c ^ (((k >> 2) & 1) << 3): a fragment read takes k-rows k and k + 4 in the two
// half-waves, which then fall 32 floats apart, in disjoint bank halves.
template <int ROWS>
struct DmaTileKOuter {
  static constexpr int BK = 32;
  static constexpr int FLOATS = ROWS * BK;
  static_assert(ROWS % 64 == 0, "k-rows of at least 16 chunks");
  __device__ static __forceinline__ int swz(int k, int pos) { return pos ^ (((k >> 2) & 1) << 3); }
  __device__ static __forceinline__ float at(const float* lds, int k, int row) {
    return lds[k * ROWS + (swz(k, row >> 2) << 2) + (row & 3)];
  }
  // k .. k+3 of one row
  __device__ static __forceinline__ f32x4 frag(const float* lds, int row, int k) {
    f32x4 v;
    v[0] = at(lds, k, row);
    v[1] = at(lds, k + 1, row);
    v[2] = at(lds, k + 2, row);
    v[3] = at(lds, k + 3, row);
    return v;
  }
};

// The MFMA work of one 32-wide K tile, cut into NB blocks.  The main loop reads a block's
// operand fragments from LDS while the previous block's MFMAs run, also across the K tiles.
template <class Cfg, class TA, class TB, class E>
struct MmaBlocks;

// fp32: four blocks of 8 k, each 4 MFMA steps of 32x32x2 on every 32x32 fragment of the wave.
template <class Cfg, class TA, class TB>
struct MmaBlocks<Cfg, TA, TB, f32x16> {
  static constexpr int NB = 4;
  struct Frag {
    f32x4 a[Cfg::FM], b[Cfg::FN];
  };
  __device__ static __forceinline__ void load(const float* As, const float* Bs, int blk, int wm0, int wn0,
                                              int lane, Frag& f) {
    const int lr = lane & 31, k = blk * 8 + (lane >> 5) * 4;
#pragma unroll
    for (int fm = 0; fm < Cfg::FM; ++fm) f.a[fm] = TA::frag(As, wm0 + fm * 32 + lr, k);
#pragma unroll
    for (int fn = 0; fn < Cfg::FN; ++fn) f.b[fn] = TB::frag(Bs, wn0 + fn * 32 + lr, k);
  }
  __device__ static __forceinline__ void mma(const Frag& f, f32x16 (&acc)[Cfg::FM][Cfg::FN]) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < Cfg::FN; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x2f32(f.a[fm][t], f.b[fn][t], acc[fm][fn], 0, 0, 0);
  }
};

// Two accumulators per 32x32 fragment, taking alternate MFMA steps (k = 2j into v[0], 2j + 1
// into v[1]), summed by the caller after the loop: a wave with one fragment then has two
// independent MFMA chains instead of one.
struct DualAcc {
  f32x16 v[2];
};

template <class Cfg, class TA, class TB>
struct MmaBlocks<Cfg, TA, TB, DualAcc> {
  static constexpr int NB = 4;
  using Frag = typename MmaBlocks<Cfg, TA, TB, f32x16>::Frag;
  __device__ static __forceinline__ void load(const float* As, const float* Bs, int blk, int wm0, int wn0,
                                              int lane, Frag& f) {
    MmaBlocks<Cfg, TA, TB, f32x16>::load(As, Bs, blk, wm0, wn0, lane, f);
  }
  __device__ static __forceinline__ void mma(const Frag& f, DualAcc (&acc)[Cfg::FM][Cfg::FN]) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int fm = 0; fm < Cfg::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < Cfg::FN; ++fn)
          acc[fm][fn].v[t & 1] =
              __builtin_amdgcn_mfma_f32_32x32x2f32(f.a[fm][t], f.b[fn][t], acc[fm][fn].v[t & 1], 0, 0, 0);
  }
};

// fp64 (pre-activations of the forward pass): two blocks of 16 k, each 4 MFMA steps of
// 16x16x4 f64 on the fp32 tile values widened exactly.
template <class Cfg, class TA, class TB>
struct MmaBlocks<Cfg, TA, TB, f64x4> {
  static constexpr int NB = 2;
  struct Frag {
    f32x4 a[Cfg::FM16], b[Cfg::FN16];
  };
  __device__ static __forceinline__ void load(const float* As, const float* Bs, int blk, int wm0, int wn0,
                                              int lane, Frag& f) {
    const int lr = lane & 15, k = blk * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int fm = 0; fm < Cfg::FM16; ++fm) f.a[fm] = TA::frag(As, wm0 + fm * 16 + lr, k);
#pragma unroll
    for (int fn = 0; fn < Cfg::FN16; ++fn) f.b[fn] = TB::frag(Bs, wn0 + fn * 16 + lr, k);
  }
  // The widening conversions of the whole block come first, so that the MFMAs issue back to
  // back instead of each waiting on the VALU conversion just before it.
  __device__ static __forceinline__ void mma(const Frag& f, f64x4 (&acc)[Cfg::FM16][Cfg::FN16]) {
    double a[Cfg::FM16][4], b[Cfg::FN16][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int fm = 0; fm < Cfg::FM16; ++fm) a[fm][t] = (double)f.a[fm][t];
#pragma unroll
      for (int fn = 0; fn < Cfg::FN16; ++fn) b[fn][t] = (double)f.b[fn][t];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int fm = 0; fm < Cfg::FM16; ++fm)
#pragma unroll
        for (int fn = 0; fn < Cfg::FN16; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[fm][t], b[fn][t], acc[fm][fn], 0, 0, 0);
  }
};

// s_waitcnt immediate (gfx9 encoding) that waits until at most n vector-memory operations of
// this wave are outstanding and does not wait on the other counters.
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
  // the count must be an immediate: the few cases the pipeline needs
  if (n <= 0) __builtin_amdgcn_s_waitcnt(0x0F70);
  else if (n == 2) __builtin_amdgcn_s_waitcnt(0x0F72);
  else if (n == 4) __builtin_amdgcn_s_waitcnt(0x0F74);
  else if (n == 8) __builtin_amdgcn_s_waitcnt(0x0F78);
  else __builtin_amdgcn_s_waitcnt(0x0F70);
}

// The same, and also until every LDS read of this wave has returned (lgkmcnt 0).
__device__ __forceinline__ void wait_vmcnt_lgkm0_dyn(int n) {
  if (n <= 0) __builtin_amdgcn_s_waitcnt(0x0070);
  else if (n == 2) __builtin_amdgcn_s_waitcnt(0x0072);
  else if (n == 4) __builtin_amdgcn_s_waitcnt(0x0074);
  else if (n == 8) __builtin_amdgcn_s_waitcnt(0x0078);
  else __builtin_amdgcn_s_waitcnt(0x0070);
}

template <class Cfg, int NSTAGE = kDmaStages>
constexpr int gemm_dma_smem_bytes() {
  return NSTAGE * (DmaTile<Cfg::BM>::FLOATS + DmaTile<Cfg::BN>::FLOATS) * 4;
}

// Buffer resource (V#) of a raw byte range: base address, stride 0, num_records = `bytes`
// (a load at or past it reads zeros), 32-bit data format.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// One 16-byte load per lane into LDS: lane l writes bytes [16 l, 16 l + 16) at `lds`, read
// from byte offset voff + soff of the resource.
__device__ __forceinline__ void buffer_dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                             float* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, soff, 0, 0);
}

// An operand of the direct-to-LDS loop is an "issuer": prepare(row0, wave, lane) once per
// tile, then issue<WAVES>(k0, lds, wave, lane) per K tile, OPS<WAVES> instructions per wave.
// DmaRowMajor: a K-contiguous row-major operand (the rows clamped to the last one), loaded by
// WAVES waves, 8 rows per instruction.  The resource starts at the tile's first row; each
// lane's byte offset inside it is fixed for the tile and the K position is the scalar offset.
template <int ROWS, int WAVES>
struct DmaRowMajor {
  using Tile = DmaTile<ROWS>;
  static_assert(ROWS % (8 * WAVES) == 0, "tile rows must split over the waves");
  static constexpr int NI = ROWS / (8 * WAVES);
  template <int WV>
  static constexpr int OPS = ROWS / (8 * WV);
  const float* __restrict__ p;
  long long ld;
  int rows;
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t voff[NI];
  __device__ __forceinline__ void prepare(int row0, int wave, int lane) {
    const int span = min(rows - row0, ROWS);
    rsrc = buffer_rsrc(p + (long long)row0 * ld, (uint32_t)((long long)span * ld * 4));
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = (i * WAVES + wave) * 8 + (lane >> 3);
      const int c = Tile::swz(r, lane & 7);                  // global chunk stored at lane & 7
      const int gr = min(r, span - 1);
      voff[i] = (uint32_t)(((long long)gr * ld + 4 * c) * 4);
    }
  }
  template <int WV>
  __device__ __forceinline__ void issue(int k0, float* lds, int wave, int) const {
    static_assert(WV == WAVES, "issuer built for this workgroup shape");
#pragma unroll
    for (int i = 0; i < NI; ++i)
      buffer_dma16(rsrc, voff[i], (uint32_t)k0 * 4u,
                   lds + __builtin_amdgcn_readfirstlane((i * WAVES + wave) * 8 * Tile::BK));
  }
};

// DmaKOuterRowMajor: a K-outer operand B[k][n] = p[k ld + n] (row k of a row-major matrix holds
// the tile's rows n0 .. n0 + ROWS - 1 at one k), in the DmaTileKOuter layout: the K tile's 32
// k-rows of ROWS floats, 16-byte chunks, loaded by WAVES waves.  Columns past `cols` are read from
// the last four (clamped; they only feed discarded outputs); the host checks cols % 4 == 0,
// 16-byte alignment, K % 32 == 0 and krows * ld * 4 < 2^31.
template <int ROWS, int WAVES>
struct DmaKOuterRowMajor {
  using Tile = DmaTileKOuter<ROWS>;
  static_assert(ROWS % (8 * WAVES) == 0, "tile rows must split over the waves");
  static constexpr int NI = ROWS / (8 * WAVES);
  template <int WV>
  static constexpr int OPS = ROWS / (8 * WV);
  const float* __restrict__ p;
  long long ld;
  int cols, krows;
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t voff[NI];
  __device__ __forceinline__ void prepare(int n0, int wave, int lane) {
    rsrc = buffer_rsrc(p, (uint32_t)((long long)krows * ld * 4));
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int o = (i * WAVES + wave) * 256 + 4 * lane;     // float offset in the tile
      const int k = o / ROWS, pos = (o % ROWS) >> 2;
      const int n = min(n0 + 4 * Tile::swz(k, pos), cols - 4);
      voff[i] = (uint32_t)(((long long)k * ld + n) * 4);
    }
  }
  template <int WV>
  __device__ __forceinline__ void issue(int k0, float* lds, int wave, int) const {
    static_assert(WV == WAVES, "issuer built for this workgroup shape");
#pragma unroll
    for (int i = 0; i < NI; ++i)
      buffer_dma16(rsrc, voff[i], (uint32_t)((long long)k0 * ld * 4),
                   lds + __builtin_amdgcn_readfirstlane((i * WAVES + wave) * 256));
  }
};

// Host check of the resource limit: a tile of `rows` rows of stride `ld` floats, read up to
// column K, spans less than 2 GiB.
__host__ inline bool dma_span_ok(long long ld, long long K, int rows) {
  return (long long)rows * ld * 4 + K * 4 < (1LL << 31);
}

// K loop over [k_begin, k_end) (k_begin a multiple of 32; a ragged last K tile is the issuers'
// business) for the tile (m0, n0), with NSTAGE LDS stages (tiles kt+1 .. kt+NSTAGE-1 in flight
// during tile kt).  One barrier per K tile, placed before the tile's last MFMA
// block: by then every wave holds that block's fragments in registers (so the stage may be
// overwritten afterwards) and has seen its own loads of tile kt+1 land, and the fragments of
// tile kt+1's first block are read while the last block's MFMAs run.  Ends with a barrier, so
// the caller may reuse `smem` afterwards.  `wave` is the wave's index among the Cfg::WAVES waves
// that share this loop and its LDS stages (the _w form lets a workgroup run several such groups,
// each on its own K range and LDS, as long as every group makes the same number of K tiles: the
// barriers are the workgroup's).
template <class Cfg, int NSTAGE, class IA, class IB, class AccT>
__device__ __forceinline__ void gemm_mainloop_dma_ops_w(IA& ia, IB& ib, int m0, int n0, int k_begin, int k_end,
                                                        float* smem, AccT& acc, int wave, int lane) {
  static_assert(Cfg::BK == 32, "direct-to-LDS main loop uses BK = 32");
  using TA = typename IA::Tile;
  using TB = typename IB::Tile;
  using MB = MmaBlocks<Cfg, TA, TB, std::remove_all_extents_t<AccT>>;
  static_assert(MB::NB % 2 == 0, "fragment buffers alternate within a K tile");
  constexpr int STAGE = TA::FLOATS + TB::FLOATS;
  constexpr int PER_TILE = IA::template OPS<Cfg::WAVES> + IB::template OPS<Cfg::WAVES>;  // DMA ops per wave
  const int wm0 = (wave / Cfg::WAVES_N) * Cfg::WM;
  const int wn0 = (wave % Cfg::WAVES_N) * Cfg::WN;
  const int nk = (k_end - k_begin + 31) / 32;
  if (nk <= 0) return;
  static_assert(NSTAGE >= 2 && NSTAGE <= 4, "two to four LDS stages");
  ia.prepare(m0, wave, lane);
  ib.prepare(n0, wave, lane);
  // tile kt lives in stage kt % NSTAGE; the K loop is unrolled NSTAGE times so that every stage
  // offset is a compile-time constant (the fragment reads then take it as an immediate offset
  // instead of recomputing their addresses at every K tile)
  auto issue = [&](int kt, float* st) {
    ia.template issue<Cfg::WAVES>(k_begin + kt * 32, st, wave, lane);
    ib.template issue<Cfg::WAVES>(k_begin + kt * 32, st + TA::FLOATS, wave, lane);
  };
  // tiles 0 .. NSTAGE - 2 in flight
  const int pre = nk < NSTAGE - 1 ? nk : NSTAGE - 1;
  for (int j = 0; j < pre; ++j) issue(j, smem + j * STAGE);
  // tile 0 in LDS (the later tiles' loads may stay in flight: loads complete in order); a bare
  // s_barrier (no fence, which would drain every outstanding load) makes it visible to every wave
  wait_vmcnt_dyn((pre - 1) * PER_TILE);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  typename MB::Frag f[2];
  MB::load(smem, smem + TA::FLOATS, 0, wm0, wn0, lane, f[0]);
  auto tile = [&](int kt, auto stage_tag) {
    constexpr int S = decltype(stage_tag)::value;
    const float* st = smem + S * STAGE;
    if (kt + NSTAGE - 1 < nk) issue(kt + NSTAGE - 1, smem + ((S + NSTAGE - 1) % NSTAGE) * STAGE);
#pragma unroll
    for (int blk = 0; blk + 1 < MB::NB; ++blk) {
      MB::load(st, st + TA::FLOATS, blk + 1, wm0, wn0, lane, f[(blk + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
      MB::mma(f[blk & 1], acc);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (kt + 1 < nk) {
      // this wave's loads of tile kt+1 landed (those of tiles kt+2 .. kt+NSTAGE-1 may stay in
      // flight) and its reads of tile kt returned; after the barrier every wave's have
      const int later = nk - kt - 2 < NSTAGE - 2 ? nk - kt - 2 : NSTAGE - 2;
      wait_vmcnt_lgkm0_dyn((later > 0 ? later : 0) * PER_TILE);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      const float* sn = smem + ((S + 1) % NSTAGE) * STAGE;
      MB::load(sn, sn + TA::FLOATS, 0, wm0, wn0, lane, f[0]);
      __builtin_amdgcn_sched_barrier(0);
    }
    MB::mma(f[(MB::NB - 1) & 1], acc);
    __builtin_amdgcn_sched_barrier(0);
  };
  // whole groups of NSTAGE tiles, then the remainder (no tile of the loop body is conditional,
  // which would make the accumulators flow through two paths and be copied at every iteration)
  int kb = 0;
  for (; kb + NSTAGE <= nk; kb += NSTAGE) {
    tile(kb, std::integral_constant<int, 0>{});
    tile(kb + 1, std::integral_constant<int, 1>{});
    if constexpr (NSTAGE > 2) tile(kb + 2, std::integral_constant<int, 2>{});
    if constexpr (NSTAGE > 3) tile(kb + 3, std::integral_constant<int, 3>{});
  }
  if (kb < nk) tile(kb, std::integral_constant<int, 0>{});
  if constexpr (NSTAGE > 2)
    if (kb + 1 < nk) tile(kb + 1, std::integral_constant<int, 1>{});
  if constexpr (NSTAGE > 3)
    if (kb + 2 < nk) tile(kb + 2, std::integral_constant<int, 2>{});
  __syncthreads();
}

template <class Cfg, int NSTAGE, class IA, class IB, class AccT>
__device__ __forceinline__ void gemm_mainloop_dma_ops(IA& ia, IB& ib, int m0, int n0, int k_begin, int k_end,
                                                      float* smem, AccT& acc) {
  gemm_mainloop_dma_ops_w<Cfg, NSTAGE>(ia, ib, m0, n0, k_begin, k_end, smem, acc, (int)(threadIdx.x >> 6),
                                       (int)(threadIdx.x & 63));
}

// Both operands K-contiguous row-major (LoadKInnerT<true> conditions, K % 32 == 0).
template <class Cfg, int NSTAGE = kDmaStages, class AccT>
__device__ __forceinline__ void gemm_mainloop_dma(const float* __restrict__ A, long long lda, int rowsA,
                                                  const float* __restrict__ B, long long ldb, int rowsB,
                                                  int m0, int n0, int k_begin, int k_end, float* smem,
                                                  AccT& acc) {
  DmaRowMajor<Cfg::BM, Cfg::WAVES> ia{A, lda, rowsA};
  DmaRowMajor<Cfg::BN, Cfg::WAVES> ib{B, ldb, rowsB};
  gemm_mainloop_dma_ops<Cfg, NSTAGE>(ia, ib, m0, n0, k_begin, k_end, smem, acc);
}

}  // namespace ntk
