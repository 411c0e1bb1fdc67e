// Host-logic check of the streamed rounds' chunk packing (wl_host.h): on a
// seeded skewed graph, every needed row's entries must arrive exactly once,
// in order, inside chunk and segment bounds, and the folds of cut rows must
// reassemble their sums.  Sums of col * weight stand in for the image.
//   stream_plan_check N AVG_DEG CHUNK WEIGHTED ACT_PERCENT SEED
#include <cstdio>
#include <cstdlib>
#include <random>

#include "../../paper_2607_02603_amd/csrc/wl_host.h"

using namespace wl;

int main(int argc, char** argv) {
  if (argc < 7) return 2;
  const uint64_t n = strtoull(argv[1], nullptr, 10);
  const double avg = atof(argv[2]);
  const uint64_t mc = strtoull(argv[3], nullptr, 10);
  const bool weighted = atoi(argv[4]) != 0;
  const int act_pct = atoi(argv[5]);
  std::mt19937_64 rng(strtoull(argv[6], nullptr, 10));
  std::uniform_real_distribution<double> U(0, 1);
  std::vector<uint64_t> rp(n + 1, 0);
  for (uint64_t i = 0; i < n; ++i) {
    const double u = U(rng);
    uint64_t d = u < 0.05 ? 0 : (uint64_t)(avg * 0.05 / (u * u * u));  // heavy tail
    d = std::min<uint64_t>(d, 40 * kSegMax);
    rp[i + 1] = rp[i] + d;
  }
  const uint64_t m = rp[n];
  std::vector<uint32_t> col(m), wt(weighted ? m : 0);
  for (uint64_t e = 0; e < m; ++e) {
    col[e] = (uint32_t)(rng() % n);
    if (weighted) wt[e] = (uint32_t)(1 + rng() % 9);
  }
  HostPool pool;
  StreamPlan P;  // rebuilt for every pattern: its arrays shrink and grow
  uint64_t bad = 0;
  // the act percentage given, a third of it, then every row
  for (int pass = 0; pass < 3; ++pass) {
    const int pct = pass == 0 ? act_pct : (pass == 1 ? act_pct / 3 : 100);
    std::vector<uint8_t> act(n);
    for (uint64_t i = 0; i < n; ++i) act[i] = (int)(rng() % 100) < pct;
    HostGraph G;
    G.n = n;
    G.m = m;
    G.rp64 = rp.data();
    G.col = col.data();
    G.wt = weighted ? wt.data() : nullptr;
    if (!P.build(pool, G, act.data())) return printf("plan allocation failed\n"), 1;
    const uint64_t sc = stream_segs(mc), fc = stream_folds(mc);
    std::vector<uint32_t> node(sc), hc(mc), hw(mc);
    std::vector<uint64_t> off(sc + 1), part(sc), got(n, 0);
    std::vector<StreamFold> fold(fc);
    uint64_t a = 0, chunks = 0, cut = 0;
    while (a < P.ns) {
      const uint64_t b = P.chunk_end(a, mc, sc);
      if (b <= a || b - a > sc) return printf("bad chunk end\n"), 1;
      const int64_t nf = P.pack(pool, G, a, b, node.data(), off.data(), hc.data(),
                                weighted ? hw.data() : nullptr, fold.data(), fc);
      if (nf < 0) return printf("fold table overflow\n"), 1;
      const uint64_t nseg = b - a;
      if (off[0] != 0 || off[nseg] > mc) return printf("bad chunk length\n"), 1;
      for (uint64_t t = 0; t < nseg; ++t) {
        if (off[t + 1] <= off[t] || off[t + 1] - off[t] > kSegMax)
          return printf("bad segment\n"), 1;
        uint64_t s = 0;
        for (uint64_t e = off[t]; e < off[t + 1]; ++e)
          s += (uint64_t)hc[e] * (weighted ? hw[e] : 1);
        if (node[t] & kSegPartial) {
          part[t] = s;
          ++cut;
        } else {
          if ((node[t] & ~kSegPartial) >= n) return printf("bad node\n"), 1;
          got[node[t]] = s;
        }
      }
      for (int64_t f = 0; f < nf; ++f) {
        const StreamFold d = fold[f];
        if ((uint64_t)d.first + d.count > nseg || d.node >= n) return printf("bad fold\n"), 1;
        uint64_t s = d.add ? got[d.node] : 0;
        for (uint32_t t = 0; t < d.count; ++t) s += part[d.first + t];
        got[d.node] = s;
      }
      a = b;
      ++chunks;
    }
    uint64_t bad_p = 0, rows = 0;
    for (uint64_t i = 0; i < n; ++i) {
      uint64_t s = 0;
      if (act[i])
        for (uint64_t e = rp[i]; e < rp[i + 1]; ++e) s += (uint64_t)col[e] * (weighted ? wt[e] : 1);
      bad_p += s != got[i];
      rows += act[i] && rp[i + 1] > rp[i];
    }
    if (rows != P.nr) return printf("row count %llu, plan %llu\n", (unsigned long long)rows,
                                    (unsigned long long)P.nr), 1;
    printf("act %d%%: n=%llu m=%llu rows=%llu segments=%llu chunks=%llu cut=%llu bad=%llu\n",
           pct, (unsigned long long)n, (unsigned long long)m, (unsigned long long)P.nr,
           (unsigned long long)P.ns, (unsigned long long)chunks, (unsigned long long)cut,
           (unsigned long long)bad_p);
    bad += bad_p;
  }
  return bad ? 1 : 0;
}
