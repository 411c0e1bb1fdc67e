// Host check of the merged partition of Algorithm 2 (merge_blocks in
// wl_host.h) against the plain first-occurrence definition, on seeded key
// patterns: keys confined to contiguous node ranges (one batch each), keys
// spread over the whole array, and boundary nodes (no key) in between.
//   merge_check N NKEYS SPREAD BOUNDARY_PERCENT SEED
#include <cstdio>
#include <cstdlib>
#include <random>

#include "../../paper_2607_02603_amd/csrc/wl_host.h"

using namespace wl;

int main(int argc, char** argv) {
  if (argc < 6) return 2;
  const uint64_t n = strtoull(argv[1], nullptr, 10);
  const uint64_t nkeys = strtoull(argv[2], nullptr, 10);
  const bool spread = atoi(argv[3]) != 0;
  const int bpct = atoi(argv[4]);
  std::mt19937_64 rng(strtoull(argv[5], nullptr, 10));
  std::vector<uint32_t> key(n);
  for (uint64_t i = 0; i < n; ++i) {
    if ((int)(rng() % 100) < bpct) {
      key[i] = kNoKey;
    } else if (spread) {
      key[i] = (uint32_t)(rng() % nkeys);
    } else {
      // keys of node i drawn near i * nkeys / n: each key's nodes are close
      const uint64_t c = i * nkeys / n;
      key[i] = (uint32_t)std::min<uint64_t>(nkeys - 1, c + rng() % 3);
    }
  }
  // the definition
  std::vector<uint32_t> mapk(nkeys, kNoKey), blk_ref(n);
  std::vector<uint8_t> rep_ref(n, 0);
  uint32_t next = 0;
  for (uint64_t i = 0; i < n; ++i) {
    const uint32_t kk = key[i];
    if (kk == kNoKey) {
      rep_ref[i] = 1;
      blk_ref[i] = next++;
    } else {
      if (mapk[kk] == kNoKey) {
        mapk[kk] = next++;
        rep_ref[i] = 1;
      }
      blk_ref[i] = mapk[kk];
    }
  }
  HostPool pool;
  std::vector<uint32_t> first(nkeys), blk(n);
  std::vector<uint8_t> rep(n);
  const uint64_t nq = merge_blocks(pool, key.data(), n, nkeys, first.data(), blk.data(), rep.data());
  uint64_t bad = nq != next;
  for (uint64_t i = 0; i < n; ++i) bad += blk[i] != blk_ref[i] || rep[i] != rep_ref[i];
  printf("n=%llu keys=%llu blocks=%llu (expected %u) threads=%u bad=%llu\n",
         (unsigned long long)n, (unsigned long long)nkeys, (unsigned long long)nq, next,
         pool.size(), (unsigned long long)bad);
  return bad ? 1 : 0;
}
