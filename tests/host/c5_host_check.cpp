// Host logic of the out-of-core paths at the shape of R-MAT scale 28 with
// edge factor 32: the steps Algorithm 2 (Section 4.2) runs on the host after
// the batches of an outer iteration, and the host plan of the streamed
// rounds that the exact finish runs on the quotient.  Built with g++ under
// AddressSanitizer and UndefinedBehaviorSanitizer; no GPU.
//
//   c5_host_check N0 M0 MB MQ MC ACT_PCT SEED
//
// The input graph has N0 nodes and M0 entries, with a heavy-tailed degree
// sequence (many empty rows, hubs of up to 2^21 entries).  Its column and
// weight arrays are read-only anonymous mappings that are never written
// (every entry reads as 0): the steps checked here depend only on the row
// pointers, so entry arrays of 16e9 entries cost no memory.  Steps:
//   1. the batch cut with cap MB (and the largest cap a 32 GiB budget
//      allows), the inner rows of every batch;
//   2. a merged partition (merge_blocks) from synthetic per-batch keys, the
//      node map of the original nodes;
//   3. the quotient's chunk plan with chunks of MQ entries and the key plan
//      of every chunk; the quotient's row pointers (a block's row is its
//      representative's row, Definition "Quotient Graph");
//   4. the batch cut of the quotient and Section 5.4's early-stop test;
//   5. the streamed rounds' plan and packing of every chunk of MC entries
//      for the weighted quotient: all rows, then ACT_PCT % of the rows;
//   6. the final first-occurrence colours of the original nodes.
// Every index, offset and count is checked against a direct computation.
#include <sys/mman.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>

#include "../../paper_2607_02603_amd/csrc/wl_host.h"

using namespace wl;

namespace {

uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

#define CHECK(cond, ...)                      \
  do {                                        \
    if (!(cond)) {                            \
      printf("FAILED %s:%d: ", __FILE__, __LINE__); \
      printf(__VA_ARGS__);                    \
      printf("\n");                           \
      exit(1);                                \
    }                                         \
  } while (0)

// Read-only entry array that costs no memory: every entry reads as 0.
const uint32_t* zero_entries(uint64_t m) {
  void* p = mmap(nullptr, 4 * std::max<uint64_t>(m, 1), PROT_READ,
                 MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE, -1, 0);
  CHECK(p != MAP_FAILED, "mmap of %llu entries", (unsigned long long)m);
  return (const uint32_t*)p;
}

// Heavy-tailed degree sequence of n rows summing to exactly m: a Pareto
// tail of exponent about 2.1 (as in R-MAT and Chung-Lu graphs), a third of
// the rows empty, no row longer than 2^22 entries.
void make_row_ptr(HostPool& pool, uint64_t n, uint64_t m, uint64_t seed,
                  std::vector<uint64_t>& rp) {
  const unsigned T = pool.size();
  const double dmax = 4194304.0;
  std::vector<double> raw(n);
  std::vector<double> part(T, 0.0);
  pool.run([&](unsigned t) {
    double s = 0;
    for (uint64_t i = n * t / T; i < n * (t + 1) / T; ++i) {
      const uint64_t h = mix(seed * 0x9E3779B97F4A7C15ull + i);
      const double u = ((h >> 11) + 0.5) * (1.0 / 9007199254740992.0);
      raw[i] = u < 1.0 / 3 ? 0.0 : std::min(dmax, std::pow((1.0 - u) * 1.5, -1.0 / 1.1));
      s += raw[i];
    }
    part[t] = s;
  });
  double sum = 0;
  for (double x : part) sum += x;
  const double scale = sum > 0 ? (double)m / sum : 0.0;
  std::vector<uint64_t> d(n);
  uint64_t tot = 0;
  for (uint64_t i = 0; i < n; ++i) {
    d[i] = (uint64_t)std::min(dmax, raw[i] * scale);
    tot += d[i];
  }
  // the rounding remainder, one entry at a time over the non-empty rows
  for (uint64_t i = 0; tot < m; i = (i + 1) % n)
    if (raw[i] > 0 && d[i] < (uint64_t)dmax) {
      ++d[i];
      ++tot;
    }
  CHECK(tot == m, "degree sum");
  rp.assign(n + 1, 0);
  for (uint64_t i = 0; i < n; ++i) rp[i + 1] = rp[i] + d[i];
}

// Chunk loop of one streamed round over G with act[]: every chunk's
// segments, offsets and folds checked, the entries of every row counted.
void check_stream_round(HostPool& pool, const HostGraph& G, const uint8_t* act, uint64_t mc,
                        const char* what) {
  StreamPlan P;
  CHECK(P.build(pool, G, act), "plan allocation");
  uint64_t rows = 0, ents = 0, segs = 0;
  for (uint64_t i = 0; i < G.n; ++i)
    if (act[i] && G.rp(i + 1) > G.rp(i)) {
      ++rows;
      ents += G.rp(i + 1) - G.rp(i);
      segs += (G.rp(i + 1) - G.rp(i) + kSegMax - 1) / kSegMax;
    }
  CHECK(P.nr == rows && P.ne == ents && P.ns == segs, "plan counts %llu %llu %llu",
        (unsigned long long)P.nr, (unsigned long long)P.ne, (unsigned long long)P.ns);
  const uint64_t sc = stream_segs(mc), fc = stream_folds(mc);
  const bool weighted = G.wt != nullptr;
  std::unique_ptr<uint32_t[]> node(new uint32_t[sc]), hc(new uint32_t[mc]),
      hw(new uint32_t[weighted ? mc : 1]);
  std::unique_ptr<uint64_t[]> off(new uint64_t[sc + 1]);
  std::unique_ptr<StreamFold[]> fold(new StreamFold[fc]);
  // entries seen per row; a row's segments must add up to its length
  std::vector<uint64_t> got(G.n, 0);
  uint64_t a = 0, chunks = 0, cut = 0, total = 0, maxfold = 0;
  while (a < P.ns) {
    const uint64_t b = P.chunk_end(a, mc, sc);
    CHECK(b > a && b - a <= sc && b <= P.ns, "chunk end %llu after %llu",
          (unsigned long long)b, (unsigned long long)a);
    const int64_t nf = P.pack(pool, G, a, b, node.get(), off.get(), hc.get(),
                              weighted ? hw.get() : nullptr, fold.get(), fc);
    CHECK(nf >= 0, "fold table overflow in chunk %llu", (unsigned long long)chunks);
    const uint64_t nseg = b - a;
    CHECK(off[0] == 0 && off[nseg] <= mc && off[nseg] == P.entry_of(b) - P.entry_of(a),
          "chunk length");
    std::vector<uint8_t> in_fold(nseg, 0);
    for (int64_t f = 0; f < nf; ++f) {
      const StreamFold d = fold[f];
      CHECK((uint64_t)d.first + d.count <= nseg && d.count > 0 && d.node < G.n, "fold");
      for (uint32_t t = 0; t < d.count; ++t) {
        CHECK(!in_fold[d.first + t], "segment in two folds");
        in_fold[d.first + t] = 1;
        CHECK((node[d.first + t] & ~kSegPartial) == d.node &&
                  (node[d.first + t] & kSegPartial),
              "fold over another row");
      }
    }
    for (uint64_t t = 0; t < nseg; ++t) {
      CHECK(off[t + 1] > off[t] && off[t + 1] - off[t] <= kSegMax, "segment bounds");
      const uint32_t nd = node[t] & ~kSegPartial;
      CHECK(nd < G.n && act[nd], "segment of an unneeded row");
      CHECK(((node[t] & kSegPartial) != 0) == (bool)in_fold[t], "cut row without a fold");
      got[nd] += off[t + 1] - off[t];
      cut += (node[t] & kSegPartial) != 0;
    }
    total += off[nseg];
    maxfold = std::max<uint64_t>(maxfold, (uint64_t)nf);
    a = b;
    ++chunks;
  }
  CHECK(total == P.ne, "packed %llu of %llu entries", (unsigned long long)total,
        (unsigned long long)P.ne);
  for (uint64_t i = 0; i < G.n; ++i)
    CHECK(got[i] == (act[i] ? G.rp(i + 1) - G.rp(i) : 0), "row %llu: %llu entries packed",
          (unsigned long long)i, (unsigned long long)got[i]);
  printf("streamed %s: rows=%llu entries=%llu segments=%llu chunks=%llu cut segments=%llu "
         "max folds per chunk=%llu\n",
         what, (unsigned long long)P.nr, (unsigned long long)P.ne, (unsigned long long)P.ns,
         (unsigned long long)chunks, (unsigned long long)cut, (unsigned long long)maxfold);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc < 8) return 2;
  const uint64_t n0 = strtoull(argv[1], nullptr, 10);
  const uint64_t m0 = strtoull(argv[2], nullptr, 10);
  const uint64_t mb = strtoull(argv[3], nullptr, 10);
  const uint64_t mq = strtoull(argv[4], nullptr, 10);
  const uint64_t mc = strtoull(argv[5], nullptr, 10);
  const int act_pct = atoi(argv[6]);
  const uint64_t seed = strtoull(argv[7], nullptr, 10);
  CHECK(n0 > 0 && n0 < (1ull << 30) && mb > 0 && mq > 0 && mq < (1ull << 31) &&
            mc >= kSegMax,
        "arguments");
  HostPool pool;

  // ---- the input graph G_0 (unweighted, as the R-MAT input)
  std::vector<uint64_t> rp0;
  make_row_ptr(pool, n0, m0, seed, rp0);
  HostGraph G0;
  G0.n = n0;
  G0.m = m0;
  G0.rp64 = rp0.data();
  G0.col = zero_entries(m0);
  uint64_t maxdeg = 0, empty = 0;
  for (uint64_t i = 0; i < n0; ++i) {
    maxdeg = std::max(maxdeg, rp0[i + 1] - rp0[i]);
    empty += rp0[i + 1] == rp0[i];
  }
  printf("G0: n=%llu m=%llu max degree=%llu empty rows=%llu\n", (unsigned long long)n0,
         (unsigned long long)m0, (unsigned long long)maxdeg, (unsigned long long)empty);

  // ---- 1. batch cut and inner rows
  const std::vector<uint64_t> starts = cut_batches(G0, mb);
  const uint64_t nb = starts.size() - 1;
  CHECK(starts.front() == 0 && starts.back() == m0 && nb >= 1, "cut ends");
  for (uint64_t b = 0; b < nb; ++b) {
    CHECK(starts[b + 1] > starts[b] || m0 == 0, "empty batch");
    CHECK(starts[b + 1] - starts[b] <= mb, "batch over the cap");
  }
  std::vector<uint8_t> inner_of(n0, 0);
  std::vector<uint32_t> key(n0, kNoKey);
  uint64_t base = 0, inner_total = 0;
  for (uint64_t b = 0; b < nb; ++b) {
    uint64_t lo, hi;
    inner_rows(G0, starts, b, &lo, &hi);
    if (hi <= lo) continue;
    CHECK(rp0[lo] >= starts[b] && rp0[hi] <= starts[b + 1], "inner rows outside the batch");
    // synthetic batch refinement, shaped like R-MAT's: rows of at most one
    // entry fall into a few large classes, longer rows stay singletons
    const uint64_t nl = hi - lo, kb = 14 + nl;
    for (uint64_t i = lo; i < hi; ++i) {
      CHECK(!inner_of[i], "row inner to two batches");
      inner_of[i] = 1;
      const uint64_t d = rp0[i + 1] - rp0[i];
      key[i] = (uint32_t)(base + (d <= 1 ? 7 * d + mix(i ^ seed) % 7 : 14 + (i - lo)));
    }
    base += kb;
    inner_total += nl;
  }
  // every row not inner to a batch is a row cut by a batch boundary
  for (uint64_t i = 0; i < n0; ++i)
    if (!inner_of[i]) {
      // the batch holding the row's first entry ends inside the row
      const uint64_t b = (uint64_t)(std::upper_bound(starts.begin(), starts.end(), rp0[i]) -
                                    starts.begin()) - 1;
      CHECK(b + 1 < nb + 1 && rp0[i] < rp0[i + 1] && starts[b + 1] < rp0[i + 1],
            "row %llu is neither inner nor cut", (unsigned long long)i);
    }
  const uint64_t budget = 32ull << 30;
  auto bytes_of = [](uint64_t rows, uint64_t cap) { return 130 * rows + 12 * cap + (1u << 20); };
  const uint64_t fit = fit_batch_cap(G0, budget, bytes_of);
  CHECK(fit > 0 && bytes_of(max_inner_rows(G0, cut_batches(G0, fit)), fit) <= budget,
        "fitted cap");
  printf("batches=%llu (cap %llu), inner rows=%llu; cap fitting 32 GiB: %llu (%llu batches)\n",
         (unsigned long long)nb, (unsigned long long)mb, (unsigned long long)inner_total,
         (unsigned long long)fit, (unsigned long long)(cut_batches(G0, fit).size() - 1));

  // ---- 2. merged partition, node map
  RawBuf<uint32_t> first, blk;
  RawBuf<uint8_t> isrep;
  CHECK(first.reserve(std::max<uint64_t>(base, 1)) && blk.reserve(n0) && isrep.reserve(n0),
        "merge arrays");
  const uint64_t nq = merge_blocks(pool, key.data(), n0, base, first.p.get(), blk.p.get(),
                                   isrep.p.get());
  uint64_t reps = 0, next = 0;
  for (uint64_t i = 0; i < n0; ++i) {
    CHECK(blk[i] < nq, "block id");
    if (isrep[i]) {
      CHECK(blk[i] == next, "blocks not numbered by first occurrence");
      ++next;
      ++reps;
    }
  }
  CHECK(reps == nq, "representatives");
  std::vector<uint32_t> map0(n0);
  for (uint64_t v = 0; v < n0; ++v) map0[v] = blk[v];

  // ---- 3. quotient chunk plan and key plans; quotient row pointers
  uint64_t qcap = 0;
  for (uint64_t i = 0; i < n0; ++i)
    if (isrep[i]) qcap += rp0[i + 1] - rp0[i];
  const std::vector<QChunk> qch = quotient_chunks(G0, mq);
  CHECK(!qch.empty() && qch.front().a == 0 && qch.back().bnd == n0, "chunk cover");
  uint64_t keys = 0, long_rows = 0;
  QChunkPrep q;
  for (size_t j = 0; j < qch.size(); ++j) {
    const QChunk& c = qch[j];
    CHECK(c.bnd > c.a && (j == 0 || c.a == qch[j - 1].bnd), "chunk order");
    CHECK(c.ea == rp0[c.a] && c.ent == rp0[c.bnd] - rp0[c.a], "chunk entries");
    if (c.ent > mq) {
      CHECK(c.bnd == c.a + 1, "a chunk over the cap holds more than one row");
      ++long_rows;
      if (isrep[c.a]) keys += c.ent;
      continue;
    }
    prep_quotient_chunk(G0, c, isrep.data(), blk.data(), q);
    CHECK(q.qoff.size() == c.bnd - c.a && q.run <= c.ent && !q.qseg.empty() &&
              q.qseg.back() == q.run,
          "chunk key plan");
    for (size_t k2 = 1; k2 < q.qseg.size(); ++k2) CHECK(q.qseg[k2] > q.qseg[k2 - 1], "segments");
    keys += q.run;
  }
  CHECK(keys == qcap, "quotient keys %llu, representatives' entries %llu",
        (unsigned long long)keys, (unsigned long long)qcap);
  std::vector<uint64_t> rp1(nq + 1, 0);
  for (uint64_t i = 0; i < n0; ++i)
    if (isrep[i]) rp1[blk[i] + 1] = rp0[i + 1] - rp0[i];
  for (uint64_t b = 0; b < nq; ++b) rp1[b + 1] += rp1[b];
  CHECK(rp1[nq] == qcap, "quotient row pointers");
  printf("merged blocks=%llu; quotient: %llu entries, %zu chunks of <= %llu entries "
         "(%llu rows longer)\n",
         (unsigned long long)nq, (unsigned long long)qcap, qch.size(), (unsigned long long)mq,
         (unsigned long long)long_rows);

  // ---- 4. the quotient G_1 (weighted), its batches and the early stop
  HostGraph G1;
  G1.n = nq;
  G1.m = qcap;
  G1.rp64 = rp1.data();
  G1.col = zero_entries(qcap);
  G1.wt = zero_entries(qcap);
  const std::vector<uint64_t> starts1 = cut_batches(G1, mb);
  const bool early = starts1.size() - 1 >= nb;
  printf("quotient batches=%llu against %llu: early stop %s\n",
         (unsigned long long)(starts1.size() - 1), (unsigned long long)nb,
         early ? "fires" : "does not fire");

  // ---- 5. streamed rounds on G_1: every row, then a part of the rows
  {
    std::vector<uint8_t> act(nq, 1);
    check_stream_round(pool, G1, act.data(), mc, "all rows");
    for (uint64_t i = 0; i < nq; ++i) act[i] = (int)(mix(i + 77 * seed) % 100) < act_pct;
    check_stream_round(pool, G1, act.data(), mc, "part of the rows");
  }

  // ---- 6. final colours of the original nodes
  {
    std::vector<uint32_t> col_f(nq), out(n0);
    for (uint64_t b = 0; b < nq; ++b) col_f[b] = (uint32_t)(mix(b) % (nq / 3 + 1));
    uint32_t k = 0;
    canonical_colours(map0, col_f.data(), nq, out.data(), &k);
    uint32_t seen = 0;
    for (uint64_t v = 0; v < n0; ++v) {
      CHECK(out[v] <= seen, "colours not by first occurrence");
      if (out[v] == seen) ++seen;
    }
    CHECK(seen == k, "colour count");
    printf("final colours: %u\n", k);
  }
  printf("ok\n");
  return 0;
}
