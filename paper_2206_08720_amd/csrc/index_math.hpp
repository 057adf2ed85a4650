// index_math.hpp -- integer index arithmetic of the NTK kernels.
//
// Everything here is plain integer arithmetic compiled for both the device (the kernels) and
// the host, so that a host program can check it exhaustively on the CPU: the multiply-high
// division, the tile orders and the work ranges of the persistent (stream-K) contraction.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ntk {

// Division of non-negative int32 values by a runtime divisor via a multiply-high:
// with s = ceil(log2 d) and m = floor(2^32 (2^s - d) / d) + 1,  n / d = (umulhi(n, m) + n) >> s
// for 0 <= n < 2^31 (the round-up reciprocal method of Granlund and Montgomery, 1994).  The
// host branch performs the same 32-bit operations, wrap-around included.
struct FastDiv {
  uint32_t d = 1, m = 1, s = 0;
  FastDiv() = default;
  __host__ explicit FastDiv(uint32_t div) : d(div) {
    s = 0;
    while ((1ull << s) < d) ++s;
    m = (uint32_t)((((1ull << s) - d) << 32) / d + 1);
  }
  __host__ __device__ __forceinline__ uint32_t div(uint32_t n) const {
#if defined(__HIP_DEVICE_COMPILE__)
    return (__umulhi(n, m) + n) >> s;
#else
    return ((uint32_t)(((uint64_t)n * m) >> 32) + n) >> s;
#endif
  }
};

// Tile index -> (tm, tn).  Symmetric: enumerate the upper triangle tm <= tn row by row.
__host__ __device__ inline void tri_index(int t, int nt, int& tm, int& tn) {
  int r = 0, base = 0;
  while (base + (nt - r) <= t) {
    base += nt - r;
    ++r;
  }
  tm = r;
  tn = r + (t - base);
}

// Tile at position `ord` of the column-banded order (non-symmetric: 8 bands of
// ceil(tiles_n / 8) columns, band by band, row by row inside a band), or of the triangle order.
__host__ __device__ inline void tile_coords(int ord, int symmetric, int tiles_m, int tiles_n, int& tm,
                                            int& tn) {
  if (symmetric) {
    tri_index(ord, tiles_n, tm, tn);
    return;
  }
  const int cb = (tiles_n + 7) / 8;               // band width (columns)
  const int full = tiles_m * cb;                   // tiles in a full band
  const int band = ord / full;
  const int rem = ord - band * full;
  const int left = tiles_n - band * cb;
  const int w = left < cb ? left : cb;             // width of this band (last may be narrower)
  tm = rem / w;
  tn = band * cb + (rem - tm * w);
}

// Start of stream-K range `lam` when U units are cut into P equal contiguous ranges.
__host__ __device__ inline long long sk_start(int lam, long long U, int P) {
  return (long long)lam * U / P;
}

// The share of XCD x (of 8) in a persistent launch of P8 workgroups per XCD over T tiles of
// L layers each: tile ordinals [base, base + count), of which the first rounds * P8 are taken
// whole (data-parallel rounds) and the rest, from first_sk on, are cut into U = (tile, layer)
// units split into P8 stream-K ranges.
struct SkShare {
  int base, count, rounds, first_sk;
  long long U;
};
__host__ __device__ inline SkShare sk_share(int x, int T, int P8, int L) {
  SkShare s;
  s.base = (int)((long long)x * T / 8);
  s.count = (int)((long long)(x + 1) * T / 8) - s.base;
  s.rounds = s.count / P8;
  s.first_sk = s.base + s.rounds * P8;
  s.U = (long long)(s.count - s.rounds * P8) * L;
  return s;
}

// Partial-buffer slot that range [beg, end) writes a split tile ts to: 0 for the tile the
// range starts in, 1 for any later one (a range splits at most its first and last tiles).
__host__ __device__ inline int sk_slot(long long beg, int L, int ts) {
  return (beg / L == ts) ? 0 : 1;
}

// Tile (relative to first_sk) whose partial sums the fixup workgroup of boundary j
// (1 <= j < P8) adds up, or -1: the boundary must fall strictly inside a tile and be the
// first boundary inside it.
__host__ __device__ inline int sk_fixup_tile(const SkShare& s, int j, int P8, int L) {
  const long long b = sk_start(j, s.U, P8);
  if (b >= s.U || b % L == 0) return -1;
  const int ts = (int)(b / L);
  if (sk_start(j - 1, s.U, P8) > (long long)ts * L) return -1;
  return ts;
}

// Per-sample tile grids on 8 XCDs: workgroup ids are dispatched round robin over the XCDs, so
// workgroup id runs on XCD id % 8.  Sample s is given to XCD s % 8, and the XCD's workgroups
// take its samples one after another, all `tiles` tiles of a sample in order, so the tiles that
// share a sample's operands share that XCD's L2.  The grid has 8 * ceil(samples / 8) * tiles
// workgroups; returns false (no work) for the ids of samples past the end.
__host__ __device__ inline bool xcd_sample_tile(int id, int tiles, int samples, int& s, int& t) {
  const int xcd = id & 7, slot = id >> 3;
  const int j = slot / tiles;
  t = slot - j * tiles;
  s = j * 8 + xcd;
  return s < samples;
}

// Blocks in contiguous ranges per XCD: workgroup id runs on XCD id % 8, and XCD x takes the
// blocks [x * nblocks / 8, (x + 1) * nblocks / 8) in order, so the blocks of one XCD are
// neighbours in the caller's block order (and share that XCD's L2 for the operands they have in
// common).  The grid has 8 * ceil(nblocks / 8) workgroups; returns false for the ids past the end
// of their XCD's range.
__host__ __device__ inline bool xcd_block(int id, int nblocks, int& blk) {
  const int xcd = id & 7, slot = id >> 3;
  const int base = (int)((long long)xcd * nblocks / 8);
  const int end = (int)((long long)(xcd + 1) * nblocks / 8);
  blk = base + slot;
  return blk < end;
}

}  // namespace ntk
