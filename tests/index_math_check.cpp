// Host-side exhaustive check of the kernels' integer index arithmetic (index_math.hpp): the
// same functions the kernels call, compiled for the CPU.  Prints one line per check and exits
// non-zero on the first failure.
//
//   * FastDiv matches integer division for every divisor the kernels can meet;
//   * the triangle and column-banded tile orders are bijections onto their tile sets;
//   * the persistent contraction schedule (data-parallel rounds + stream-K ranges + fixup)
//     covers every (tile, layer) unit exactly once, writes each finished tile exactly once,
//     never writes a partial-buffer slot twice, and its fixup reads exactly the slots that
//     hold the split tile's partial sums, each layer once.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <set>
#include <utility>
#include <vector>

#include "index_math.hpp"

using namespace ntk;

#define CHECK(cond, ...)                        \
  do {                                          \
    if (!(cond)) {                              \
      std::printf("FAIL %s:%d: ", __FILE__, __LINE__); \
      std::printf(__VA_ARGS__);                 \
      std::printf("\n");                        \
      std::exit(1);                             \
    }                                           \
  } while (0)

static void check_fastdiv() {
  std::mt19937_64 rng(12345);
  std::vector<uint32_t> divs;
  for (uint32_t d = 1; d <= 5000; ++d) divs.push_back(d);
  for (int i = 0; i < 2000; ++i) divs.push_back(1 + (uint32_t)(rng() % 0x7fffffffu));
  for (int k = 12; k < 31; ++k) {
    divs.push_back(1u << k);
    divs.push_back((1u << k) - 1);
    divs.push_back((1u << k) + 1);
  }
  long long tested = 0;
  for (uint32_t d : divs) {
    const FastDiv f(d);
    auto one = [&](uint32_t n) {
      CHECK(f.div(n) == n / d, "FastDiv(%u).div(%u) = %u, expected %u", d, n, f.div(n), n / d);
      ++tested;
    };
    for (uint32_t n = 0; n < 2048; ++n) one(n);
    for (int i = 0; i < 2000; ++i) one((uint32_t)(rng() & 0x7fffffffu));
    // around multiples of d, up to the top of the int32 range
    for (int i = 0; i < 200; ++i) {
      const uint64_t q = rng() % (0x7fffffffull / d + 1);
      for (int64_t off = -1; off <= 1; ++off) {
        const int64_t n = (int64_t)(q * d) + off;
        if (n >= 0 && n <= 0x7fffffff) one((uint32_t)n);
      }
    }
    one(0x7fffffffu);
  }
  std::printf("fastdiv: %zu divisors, %lld quotients\n", divs.size(), tested);
}

static void check_tile_orders() {
  long long n = 0;
  for (int nt = 1; nt <= 160; ++nt) {
    const int T = nt * (nt + 1) / 2;
    std::vector<int> seen(nt * nt, 0);
    for (int t = 0; t < T; ++t) {
      int tm, tn;
      tile_coords(t, 1, nt, nt, tm, tn);
      CHECK(0 <= tm && tm <= tn && tn < nt, "triangle order nt=%d t=%d -> (%d,%d)", nt, t, tm, tn);
      CHECK(!seen[tm * nt + tn]++, "triangle order nt=%d visits (%d,%d) twice", nt, tm, tn);
      ++n;
    }
  }
  for (int tm_ = 1; tm_ <= 48; ++tm_)
    for (int tn_ = 1; tn_ <= 48; ++tn_) {
      std::vector<int> seen(tm_ * tn_, 0);
      const int cb = (tn_ + 7) / 8;
      for (int t = 0; t < tm_ * tn_; ++t) {
        int tm, tn;
        tile_coords(t, 0, tm_, tn_, tm, tn);
        CHECK(0 <= tm && tm < tm_ && 0 <= tn && tn < tn_, "banded order %dx%d t=%d -> (%d,%d)", tm_,
              tn_, t, tm, tn);
        CHECK(!seen[tm * tn_ + tn]++, "banded order %dx%d visits (%d,%d) twice", tm_, tn_, tm, tn);
        // band by band: ordinal t lies in band t / (tm_ * cb)
        CHECK(tn / cb == t / (tm_ * cb), "banded order %dx%d t=%d in band %d", tm_, tn_, t, tn / cb);
        ++n;
      }
    }
  std::printf("tile orders: %lld tiles\n", n);
}

// Simulate one persistent launch exactly as the contraction kernel and its fixup walk it.
static void check_schedule(int T, int P, int L) {
  const int P8 = P / 8;
  std::vector<int> units((size_t)T * L, 0), written(T, 0), fixed(T, 0), split(T, 0);
  // (owner, slot) -> (tile ordinal, l0, l1)
  std::map<std::pair<int, int>, std::vector<int>> slots;
  std::vector<int> dp_seen(T, 0);
  for (int bid = 0; bid < P; ++bid) {
    const int x = bid & 7, j = bid >> 3, lam = x * P8 + j;
    const SkShare sh = sk_share(x, T, P8, L);
    for (int i = 0; i < sh.rounds; ++i) {
      const int t = sh.base + i * P8 + j;
      CHECK(t >= sh.base && t < sh.first_sk, "T=%d P=%d L=%d: round tile %d outside share", T, P, L, t);
      for (int l = 0; l < L; ++l) ++units[(size_t)t * L + l];
      ++written[t];
    }
    const long long beg = sk_start(j, sh.U, P8), end = sk_start(j + 1, sh.U, P8);
    for (long long u = beg; u < end;) {
      const int ts = (int)(u / L);
      const int l0 = (int)(u - (long long)ts * L);
      const int l1 = (int)((long long)L < l0 + (end - u) ? (long long)L : l0 + (end - u));
      const int t = sh.first_sk + ts;
      CHECK(t < sh.base + sh.count, "T=%d P=%d L=%d: stream-K tile %d outside share", T, P, L, t);
      for (int l = l0; l < l1; ++l) ++units[(size_t)t * L + l];
      if (l0 == 0 && l1 == L) {
        ++written[t];
      } else {
        split[t] = 1;
        const auto key = std::make_pair(lam, sk_slot(beg, L, ts));
        CHECK(!slots.count(key), "T=%d P=%d L=%d: partial slot (%d,%d) written twice", T, P, L, key.first,
              key.second);
        slots[key] = {t, l0, l1};
      }
      u += l1 - l0;
    }
  }
  // fixup: one workgroup per (x, j = 1..P8-1)
  for (int blk = 0; blk < 8 * (P8 - 1); ++blk) {
    const int x = blk / (P8 - 1), j = blk % (P8 - 1) + 1;
    const SkShare sh = sk_share(x, T, P8, L);
    const int ts = sk_fixup_tile(sh, j, P8, L);
    if (ts < 0) continue;
    const int t = sh.first_sk + ts;
    ++fixed[t];
    std::vector<int> layer(L, 0);
    const long long tile_end = (long long)(ts + 1) * L;
    for (int q = j - 1; q < P8 && sk_start(q, sh.U, P8) < tile_end; ++q) {
      const long long qb = sk_start(q, sh.U, P8);
      if (sk_start(q + 1, sh.U, P8) <= qb) continue;
      const auto key = std::make_pair(x * P8 + q, sk_slot(qb, L, ts));
      auto it = slots.find(key);
      CHECK(it != slots.end(), "T=%d P=%d L=%d: fixup of tile %d reads unwritten slot (%d,%d)", T, P, L,
            t, key.first, key.second);
      CHECK(it->second[0] == t, "T=%d P=%d L=%d: fixup of tile %d reads slot of tile %d", T, P, L, t,
            it->second[0]);
      for (int l = it->second[1]; l < it->second[2]; ++l) ++layer[l];
    }
    for (int l = 0; l < L; ++l)
      CHECK(layer[l] == 1, "T=%d P=%d L=%d: fixup of tile %d sums layer %d %d times", T, P, L, t, l,
            layer[l]);
  }
  for (int t = 0; t < T; ++t) {
    for (int l = 0; l < L; ++l)
      CHECK(units[(size_t)t * L + l] == 1, "T=%d P=%d L=%d: unit (%d,%d) covered %d times", T, P, L, t, l,
            units[(size_t)t * L + l]);
    if (split[t])
      CHECK(written[t] == 0 && fixed[t] == 1, "T=%d P=%d L=%d: split tile %d written %d, fixed %d", T, P,
            L, t, written[t], fixed[t]);
    else
      CHECK(written[t] == 1 && fixed[t] == 0, "T=%d P=%d L=%d: tile %d written %d, fixed %d", T, P, L, t,
            written[t], fixed[t]);
  }
}

// every (sample, tile) exactly once, every workgroup of sample s on XCD s % 8, and an XCD's
// workgroups in sample order
static void check_xcd_sample_tile() {
  for (int samples = 1; samples <= 70; ++samples)
    for (int tiles : {1, 2, 5, 9, 45, 64}) {
      const int grid = 8 * ((samples + 7) / 8) * tiles;
      std::vector<int> seen((size_t)samples * tiles, 0);
      std::vector<int> last(8, -1);
      for (int id = 0; id < grid; ++id) {
        int s = -1, t = -1;
        if (!ntk::xcd_sample_tile(id, tiles, samples, s, t)) {
          CHECK(s >= samples, "xcd_sample_tile: id %d refused but s = %d", id, s);
          continue;
        }
        CHECK(t >= 0 && t < tiles && s >= 0, "xcd_sample_tile: id %d -> (%d, %d)", id, s, t);
        CHECK(s % 8 == id % 8, "xcd_sample_tile: sample %d on XCD %d", s, id % 8);
        CHECK(s >= last[id % 8], "xcd_sample_tile: XCD %d goes back to sample %d", id % 8, s);
        last[id % 8] = s;
        ++seen[(size_t)s * tiles + t];
      }
      for (size_t i = 0; i < seen.size(); ++i)
        CHECK(seen[i] == 1, "xcd_sample_tile: samples=%d tiles=%d unit %zu covered %d times", samples, tiles,
              i, seen[i]);
    }
}

// The per-XCD block ranges: a grid of 8 * ceil(n / 8) workgroups visits every block exactly once,
// and the blocks of one XCD form one contiguous range in block order.
static void check_xcd_block() {
  long long launches = 0;
  std::vector<int> sizes;
  for (int n = 1; n <= 4096; ++n) sizes.push_back(n);
  for (int n : {8191, 8192, 8193, 65535, 65536, 1 << 20, (1 << 20) + 5}) sizes.push_back(n);
  for (int n : sizes) {
    const int grid = 8 * ((n + 7) / 8);
    std::vector<char> seen(n, 0);
    std::vector<int> lo(8, n), hi(8, -1);
    int visited = 0;
    for (int id = 0; id < grid; ++id) {
      int blk = -1;
      if (!xcd_block(id, n, blk)) continue;
      CHECK(blk >= 0 && blk < n, "xcd_block n=%d id=%d -> %d", n, id, blk);
      CHECK(!seen[blk]++, "xcd_block n=%d visits block %d twice", n, blk);
      const int x = id & 7;
      lo[x] = std::min(lo[x], blk);
      hi[x] = std::max(hi[x], blk);
      ++visited;
    }
    CHECK(visited == n, "xcd_block n=%d visits %d blocks", n, visited);
    for (int x = 0; x < 8; ++x)
      if (hi[x] >= 0) {
        int cnt = 0;
        for (int id = x; id < grid; id += 8) {
          int blk;
          cnt += xcd_block(id, n, blk) ? 1 : 0;
        }
        CHECK(hi[x] - lo[x] + 1 == cnt, "xcd_block n=%d: XCD %d range not contiguous", n, x);
      }
    ++launches;
  }
  std::printf("xcd_block: %lld grids\n", launches);
}

int main() {
  check_fastdiv();
  check_tile_orders();
  check_xcd_sample_tile();
  check_xcd_block();
  long long n = 0;
  const int Ps[] = {16, 24, 32, 64, 80, 128, 256, 304, 512};
  const int Ls[] = {1, 2, 3, 5, 8, 9, 17};
  for (int P : Ps)
    for (int L : Ls) {
      for (int T = 0; T <= 3 * P + 9; ++T, ++n) check_schedule(T, P, L);
      for (int T : {8 * P - 1, 8 * P, 8 * P + 1, 2080, 2145, 4096, 4097}) check_schedule(T, P, L), ++n;
    }
  std::printf("stream-K schedule: %lld launches\n", n);
  std::printf("OK\n");
  return 0;
}
