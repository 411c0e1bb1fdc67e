// Host check of Theorem 1's row-sum bound for arithmetic mod 2^64
// (ring_row_sums_ok in wl_host.h): unweighted rows by length, weighted rows
// by the sum of their weights, at and just above 2^32, on 32- and 64-bit row
// pointers, with rows spread over all pool threads.
#include <cstdio>
#include <vector>

#include "../../paper_2607_02603_amd/csrc/wl_host.h"

using namespace wl;

static int expect(bool got, bool want, const char* what) {
  if (got != want) {
    printf("FAIL %s: got %d want %d\n", what, (int)got, (int)want);
    return 1;
  }
  return 0;
}

int main() {
  HostPool pool(8);
  int bad = 0;
  // weighted: 1000 rows of 3 entries; row r sums to 2^32 (ok) or 2^32 + 1
  for (int where : {0, 517, 999}) {
    for (int over : {0, 1}) {
      const uint64_t n = 1000;
      std::vector<uint64_t> rp(n + 1);
      std::vector<uint32_t> wt(3 * n, 7);
      for (uint64_t i = 0; i <= n; ++i) rp[i] = 3 * i;
      wt[3 * where] = 1u << 31;
      wt[3 * where + 1] = (1u << 31) - 1;
      wt[3 * where + 2] = 1 + over;
      HostGraph G;
      G.n = n;
      G.m = 3 * n;
      G.rp64 = rp.data();
      G.wt = wt.data();
      bad += expect(ring_row_sums_ok(pool, G), !over, "weighted");
    }
  }
  // unweighted: a row of length 2^32 + 1 through 32-bit row pointers is not
  // representable; a 64-bit row pointer with such a row (no entries read)
  for (uint64_t len : {(1ull << 32), (1ull << 32) + 1}) {
    std::vector<uint64_t> rp = {0, 5, 5 + len, 5 + len + 2};
    HostGraph G;
    G.n = 3;
    G.m = rp[3];
    G.rp64 = rp.data();
    bad += expect(ring_row_sums_ok(pool, G), len == (1ull << 32), "unweighted 64");
  }
  {
    std::vector<uint32_t> rp = {0, 4, 4, 9};
    HostGraph G;
    G.n = 3;
    G.m = 9;
    G.rp32 = rp.data();
    bad += expect(ring_row_sums_ok(pool, G), true, "unweighted 32");
  }
  printf(bad ? "failures: %d\n" : "ok\n", bad);
  return bad ? 1 : 0;
}
