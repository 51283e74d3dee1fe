// Checks ms::GatherPool on the host: every thread count splits the rows
// exactly, ids outside the store give zero rows, and a pool is reusable.
#include <cstdio>
#include <cstring>
#include <vector>

#include "../../paper_2410_22697_amd/csrc/gather_pool.hpp"

int main() {
  const int64_t nrows = 1000, rb = 20;
  std::vector<uint8_t> store(nrows * rb);
  for (int64_t i = 0; i < nrows * rb; ++i) store[i] = (uint8_t)((i * 131) % 251);
  int bad = 0;
  for (int threads : {1, 2, 3, 8}) {
    ms::GatherPool pool(threads);
    for (int64_t n : {0, 1, 7, 999, 2500}) {
      std::vector<int32_t> rows(n);
      for (int64_t i = 0; i < n; ++i) rows[i] = (int32_t)((i * 7919) % (nrows + 40)) - 20;  // some out of range
      std::vector<uint8_t> dst(n * rb + 1, 0xEE);
      pool.gather(store.data(), nrows, rb, rows.data(), n, dst.data());
      for (int64_t i = 0; i < n; ++i) {
        const int32_t r = rows[i];
        for (int64_t b = 0; b < rb; ++b) {
          const uint8_t want = (r >= 0 && r < nrows) ? store[r * rb + b] : 0;
          if (dst[i * rb + b] != want) ++bad;
        }
      }
      if (dst[n * rb] != 0xEE) ++bad;  // nothing past the n rows
    }
  }
  std::printf("mismatches %d\n", bad);
  return bad ? 1 : 0;
}
