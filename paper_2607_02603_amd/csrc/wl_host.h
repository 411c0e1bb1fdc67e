// Host-side pieces of the out-of-core paths, in plain C++ (no HIP): the
// host CSR view, a fork-join thread pool, and the packing of the rows whose
// image a streamed round needs into chunks of segments (wl_stream.h).
#pragma once
#include <sched.h>

#include <algorithm>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <functional>
#include <memory>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

namespace wl {

constexpr uint32_t kSegMax = 4096;          // entries per segment (one wave)
constexpr uint32_t kSegPartial = 1u << 31;  // node flag: partial sum of a cut row

// A CSR graph in host memory (the caller's arrays or the library's).
struct HostGraph {
  uint64_t n = 0, m = 0;
  const uint32_t* rp32 = nullptr;
  const uint64_t* rp64 = nullptr;
  const uint32_t* col = nullptr;
  const uint32_t* wt = nullptr;
  uint64_t rp(uint64_t i) const { return rp64 ? rp64[i] : (uint64_t)rp32[i]; }
  // first row i in [0, n] with rp(i) >= v
  uint64_t lower_row(uint64_t v) const {
    uint64_t lo = 0, hi = n;
    while (lo < hi) {
      uint64_t mid = (lo + hi) / 2;
      if (rp(mid) < v) lo = mid + 1; else hi = mid;
    }
    return lo;
  }
};

// Fork-join over a fixed set of host threads (the caller is thread 0).
class HostPool {
 public:
  explicit HostPool(unsigned max_threads = 16) {
    cpu_set_t set;
    CPU_ZERO(&set);
    unsigned t = 4;
    if (sched_getaffinity(0, sizeof(set), &set) == 0) t = (unsigned)CPU_COUNT(&set);
    n_ = std::max(1u, std::min(t, max_threads));
    for (unsigned i = 1; i < n_; ++i) {
      try {
        th_.emplace_back([this, i] { loop(i); });
      } catch (...) {
        n_ = i;
        break;
      }
    }
  }
  ~HostPool() {
    {
      std::lock_guard<std::mutex> g(m_);
      stop_ = true;
      ++gen_;
    }
    cv_.notify_all();
    for (auto& t : th_) t.join();
  }
  HostPool(const HostPool&) = delete;
  HostPool& operator=(const HostPool&) = delete;
  unsigned size() const { return n_; }
  // fn(i) for every i in [0, size()); returns when all have returned.
  void run(const std::function<void(unsigned)>& fn) {
    {
      std::lock_guard<std::mutex> g(m_);
      fn_ = &fn;
      pending_ = n_ - 1;
      ++gen_;
    }
    cv_.notify_all();
    fn(0);
    std::unique_lock<std::mutex> g(m_);
    done_.wait(g, [&] { return pending_ == 0; });
    fn_ = nullptr;
  }

 private:
  void loop(unsigned i) {
    uint64_t seen = 0;
    for (;;) {
      const std::function<void(unsigned)>* f;
      {
        std::unique_lock<std::mutex> g(m_);
        cv_.wait(g, [&] { return gen_ != seen; });
        seen = gen_;
        if (stop_) return;
        f = fn_;
      }
      (*f)(i);
      {
        std::lock_guard<std::mutex> g(m_);
        if (--pending_ == 0) done_.notify_one();
      }
    }
  }
  unsigned n_ = 1;
  std::vector<std::thread> th_;
  std::mutex m_;
  std::condition_variable cv_, done_;
  const std::function<void(unsigned)>* fn_ = nullptr;
  unsigned pending_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

// Theorem 1's precondition for arithmetic mod 2^64: every row sum of G at
// most 2^32 (the row length for an unweighted G).
inline bool ring_row_sums_ok(HostPool& pool, const HostGraph& G) {
  const unsigned T = pool.size();
  std::vector<uint8_t> bad(T, 0);
  pool.run([&](unsigned t) {
    for (uint64_t i = G.n * t / T; i < G.n * (t + 1) / T; ++i) {
      const uint64_t beg = G.rp(i), end = G.rp(i + 1);
      uint64_t sum = end - beg;
      if (G.wt) {
        sum = 0;
        for (uint64_t e = beg; e < end && sum <= (1ull << 32); ++e) sum += G.wt[e];
      }
      if (sum > (1ull << 32)) {
        bad[t] = 1;
        return;
      }
    }
  });
  for (unsigned t = 0; t < T; ++t)
    if (bad[t]) return false;
  return true;
}

// Growable array that is not value-initialised: a fresh allocation is first
// touched by the threads that fill it, and every slot read later has been
// written.  reserve() returns false when the allocation fails.
template <typename T>
struct RawBuf {
  std::unique_ptr<T[]> p;
  uint64_t cap = 0;
  bool reserve(uint64_t n) {
    if (n <= cap) return true;
    p.reset(new (std::nothrow) T[n]);
    cap = p ? n : 0;
    return p != nullptr;
  }
  T& operator[](uint64_t i) { return p[i]; }
  const T& operator[](uint64_t i) const { return p[i]; }
  const T* data() const { return p.get(); }
};

// f(i) for every i in [lo, hi) with act[i] != 0, reading act eight bytes at
// a time (the active rows of late rounds are few).
template <typename F>
inline void for_active(const uint8_t* act, uint64_t lo, uint64_t hi, F&& f) {
  uint64_t i = lo;
  for (; i + 8 <= hi; i += 8) {
    uint64_t w;
    memcpy(&w, act + i, 8);
    while (w) {
      const int b = __builtin_ctzll(w) >> 3;
      f(i + (uint64_t)b);
      w &= ~(0xFFull << (8 * b));
    }
  }
  for (; i < hi; ++i)
    if (act[i]) f(i);
}

// Merged partition of Algorithm 2 (Eq. merge) numbered by first occurrence
// in node order: a node whose key is kNoKey (a boundary node) is a block of
// its own, nodes sharing a key form one block.  Writes blk[i] (block of node
// i) and isrep[i] (1 for the first node of its block) and returns the
// number of blocks.  first (nkeys entries) is scratch.
constexpr uint32_t kNoKey = 0xFFFFFFFFu;

inline uint64_t merge_blocks(HostPool& pool, const uint32_t* key, uint64_t n, uint64_t nkeys,
                             uint32_t* first, uint32_t* blk, uint8_t* isrep) {
  const unsigned T = pool.size();
  auto lo = [&](unsigned t) { return n * t / T; };
  pool.run([&](unsigned t) {
    for (uint64_t k = nkeys * t / T; k < nkeys * (t + 1) / T; ++k) first[k] = kNoKey;
  });
  // first node of every key (a key's nodes rarely span two threads' ranges)
  pool.run([&](unsigned t) {
    for (uint64_t i = lo(t); i < lo(t + 1); ++i) {
      const uint32_t kk = key[i];
      if (kk == kNoKey) continue;
      uint32_t cur = __atomic_load_n(&first[kk], __ATOMIC_RELAXED);
      while ((uint32_t)i < cur &&
             !__atomic_compare_exchange_n(&first[kk], &cur, (uint32_t)i, true, __ATOMIC_RELAXED,
                                          __ATOMIC_RELAXED)) {
      }
    }
  });
  std::vector<uint64_t> cnt(T + 1, 0);
  pool.run([&](unsigned t) {
    uint64_t c = 0;
    for (uint64_t i = lo(t); i < lo(t + 1); ++i) {
      const uint32_t kk = key[i];
      c += kk == kNoKey || first[kk] == (uint32_t)i;
    }
    cnt[t + 1] = c;
  });
  for (unsigned t = 0; t < T; ++t) cnt[t + 1] += cnt[t];
  pool.run([&](unsigned t) {
    uint64_t id = cnt[t];
    for (uint64_t i = lo(t); i < lo(t + 1); ++i) {
      const uint32_t kk = key[i];
      const bool fresh = kk == kNoKey || first[kk] == (uint32_t)i;
      isrep[i] = fresh ? 1 : 0;
      if (fresh) blk[i] = (uint32_t)id++;
    }
  });
  // the other nodes take the block of their key's first node
  pool.run([&](unsigned t) {
    for (uint64_t i = lo(t); i < lo(t + 1); ++i)
      if (!isrep[i]) blk[i] = blk[first[key[i]]];
  });
  return cnt[T];
}

// Largest value v in [0, cap] with total_of(v) <= budget (total_of is
// non-decreasing), or 0.
template <typename F>
inline uint64_t largest_fitting(F total_of, uint64_t budget, uint64_t cap) {
  uint64_t lo = 0, hi = cap;
  while (lo < hi) {
    uint64_t mid = lo + (hi - lo + 1) / 2;
    if (total_of(mid) <= budget) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// Algorithm 2 (Section 4.2), host side: the batch cut, the inner rows of a
// batch, the chunk plan of the quotient and the final colours.
// ---------------------------------------------------------------------------

// Greedy batch cut of the entry array: ranges of at most mb >= 1 entries
// ending at a row boundary, a row longer than mb cut inside (reading of
// Algorithm 2's "partition E into E_1 .. E_Nb with |E_k| <= M_b").  Returns
// the starts of the ranges followed by m (at least {0, m}).
inline std::vector<uint64_t> cut_batches(const HostGraph& G, uint64_t mb) {
  std::vector<uint64_t> starts;
  uint64_t s = 0;
  const uint64_t m = G.m;
  do {
    starts.push_back(s);
    if (m - s <= mb) { s = m; break; }
    const uint64_t lim = s + mb;
    // last row boundary <= lim
    uint64_t lo = 0, hi = G.n;
    while (lo < hi) {
      uint64_t mid = lo + (hi - lo + 1) / 2;
      if (G.rp(mid) <= lim) lo = mid; else hi = mid - 1;
    }
    uint64_t e = G.rp(lo);
    if (e <= s) e = lim;
    s = e;
  } while (s < m);
  starts.push_back(m);
  return starts;
}

// Inner rows of batch b (Definition "Inner and boundary nodes"): the rows
// that start inside it and end inside it; empty rows belong to the batch
// whose range contains their offset.
inline void inner_rows(const HostGraph& G, const std::vector<uint64_t>& starts, uint64_t b,
                       uint64_t* r_lo, uint64_t* r_hi) {
  const uint64_t nb = starts.size() - 1, eb = starts[b + 1];
  *r_lo = G.lower_row(starts[b]);
  *r_hi = (b + 1 == nb) ? G.n : G.lower_row(eb);
  if (*r_hi > *r_lo && G.rp(*r_hi) > eb) --*r_hi;  // the last row continues
}

inline uint64_t max_inner_rows(const HostGraph& G, const std::vector<uint64_t>& starts) {
  uint64_t mx = 0;
  for (uint64_t b = 0; b + 1 < starts.size(); ++b) {
    uint64_t lo, hi;
    inner_rows(G, starts, b, &lo, &hi);
    if (hi > lo) mx = std::max(mx, hi - lo);
  }
  return mx;
}

// Largest batch cap whose batches fit a device budget: bytes_of(rows, cap)
// is the workspace a batch of 'rows' inner rows and 'cap' entries needs.
// Returns 0 when not even a cap of one entry fits.
template <typename F>
inline uint64_t fit_batch_cap(const HostGraph& G, uint64_t budget, F bytes_of) {
  const uint64_t mall = std::max<uint64_t>(G.m, 1);  // a cap >= m is one batch
  auto fits = [&](uint64_t cap) {
    const std::vector<uint64_t> st = cut_batches(G, cap);
    return bytes_of(max_inner_rows(G, st), cap) <= budget;
  };
  uint64_t lo = 0, hi = std::min(mall, budget / 8);
  while (lo < hi) {
    const uint64_t mid = lo + (hi - lo + 1) / 2;
    if (fits(mid)) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// A chunk of the quotient phase: rows [a, bnd) holding entries
// [ea, ea + ent).  ent <= mq, or the chunk is one row longer than mq
// (processed in pieces).
struct QChunk {
  uint64_t a, bnd, ea, ent;
};

// Row ranges of at most mq >= 1 entries (at least one row each) covering
// all n rows.
inline std::vector<QChunk> quotient_chunks(const HostGraph& G, uint64_t mq) {
  std::vector<QChunk> qch;
  const uint64_t n = G.n;
  for (uint64_t a = 0; a < n;) {
    const uint64_t ea = G.rp(a);
    uint64_t lo = a + 1, hi = n;  // last row end <= ea + mq (at least one row)
    while (lo < hi) {
      const uint64_t mid = lo + (hi - lo + 1) / 2;
      if (G.rp(mid) - ea <= mq) lo = mid; else hi = mid - 1;
    }
    qch.push_back({a, lo, ea, G.rp(lo) - ea});
    a = lo;
  }
  return qch;
}

// The key plan of one quotient chunk (ent <= mq < 2^32): for each row, the
// offset of its keys among the chunk's keys (only representatives' rows
// have keys, Definition "Quotient Graph"); the key offsets where the
// non-empty representative rows start, followed by the key count; the
// number of representatives and the block of the first one.
struct QChunkPrep {
  std::vector<uint64_t> qoff;
  std::vector<uint32_t> qseg;
  uint64_t run = 0, nreps = 0;
  uint32_t bfirst = 0xFFFFFFFFu;
};

inline void prep_quotient_chunk(const HostGraph& G, const QChunk& c, const uint8_t* isrep,
                                const uint32_t* blk, QChunkPrep& q) {
  const uint64_t nrows = c.bnd - c.a;
  q.qoff.resize(nrows);
  q.qseg.clear();
  q.run = q.nreps = 0;
  q.bfirst = 0xFFFFFFFFu;
  for (uint64_t r = 0; r < nrows; ++r) {
    q.qoff[r] = q.run;
    if (isrep[c.a + r]) {
      if (q.bfirst == 0xFFFFFFFFu) q.bfirst = blk[c.a + r];
      const uint64_t d = G.rp(c.a + r + 1) - G.rp(c.a + r);
      if (d) q.qseg.push_back((uint32_t)q.run);
      q.run += d;
      ++q.nreps;
    }
  }
  q.qseg.push_back((uint32_t)q.run);
}

// Final colours of the original nodes: the colour of the node of the last
// graph each maps to (col_f, or the node itself when col_f is NULL),
// numbered by first occurrence.  Every map0[v] < nf, every col_f[.] < nf.
inline void canonical_colours(const std::vector<uint32_t>& map0, const uint32_t* col_f,
                              uint64_t nf, uint32_t* color_out, uint32_t* k_out) {
  std::vector<uint32_t> slot(nf, 0xFFFFFFFFu);
  uint32_t k = 0;
  for (uint64_t v = 0; v < map0.size(); ++v) {
    const uint32_t c = col_f ? col_f[map0[v]] : map0[v];
    uint32_t& sl = slot[c];
    if (sl == 0xFFFFFFFFu) sl = k++;
    color_out[v] = sl;
  }
  *k_out = k;
}

// A cut row's share of one chunk: its segments [first, first + count) of the
// chunk, the node, and whether z already holds the sum of earlier chunks.
struct StreamFold {
  uint32_t first, count, node, add;
};

// Capacity of one chunk of at most mc entries.
inline uint64_t stream_segs(uint64_t mc) { return mc / 4 + 1; }
// a cut row has more than kSegMax entries: at most mc / kSegMax lie inside
// a chunk, plus the two that reach over its ends
inline uint64_t stream_folds(uint64_t mc) { return mc / kSegMax + 2; }

// The rows of one streamed round whose image is needed (act set, at least
// one entry), in node order, each cut into segments of at most kSegMax
// entries.  Segments are numbered over the round; seg0[r] / ent0[r] are the
// first segment and the first packed entry of live row r.
struct StreamPlan {
  RawBuf<uint32_t> rows;
  RawBuf<uint64_t> seg0, ent0;
  uint64_t nr = 0, ns = 0, ne = 0;

  // false when the host arrays cannot be allocated
  bool build(HostPool& pool, const HostGraph& G, const uint8_t* act) {
    const unsigned T = pool.size();
    const uint64_t n = G.n;
    std::vector<uint64_t> tc(T + 1, 0), ts(T + 1, 0), te(T + 1, 0);
    auto lo = [&](unsigned t) { return n * t / T; };
    pool.run([&](unsigned t) {
      uint64_t c = 0, sg = 0, en = 0;
      for_active(act, lo(t), lo(t + 1), [&](uint64_t i) {
        const uint64_t d = G.rp(i + 1) - G.rp(i);
        if (d == 0) return;
        ++c;
        sg += (d + kSegMax - 1) / kSegMax;
        en += d;
      });
      tc[t + 1] = c;
      ts[t + 1] = sg;
      te[t + 1] = en;
    });
    for (unsigned t = 0; t < T; ++t) {
      tc[t + 1] += tc[t];
      ts[t + 1] += ts[t];
      te[t + 1] += te[t];
    }
    nr = tc[T];
    ns = ts[T];
    ne = te[T];
    if (!rows.reserve(nr + 1) || !seg0.reserve(nr + 1) || !ent0.reserve(nr + 1)) {
      nr = ns = ne = 0;
      return false;
    }
    pool.run([&](unsigned t) {
      uint64_t c = tc[t], sg = ts[t], en = te[t];
      for_active(act, lo(t), lo(t + 1), [&](uint64_t i) {
        const uint64_t d = G.rp(i + 1) - G.rp(i);
        if (d == 0) return;
        rows[c] = (uint32_t)i;
        seg0[c] = sg;
        ent0[c] = en;
        ++c;
        sg += (d + kSegMax - 1) / kSegMax;
        en += d;
      });
    });
    seg0[nr] = ns;
    ent0[nr] = ne;
    return true;
  }

  // live row holding segment g < ns
  uint64_t row_of(uint64_t g) const {
    return (uint64_t)(std::upper_bound(seg0.data(), seg0.data() + nr, g) - seg0.data()) - 1;
  }
  // packed entry where segment g starts (ne for g >= ns)
  uint64_t entry_of(uint64_t g) const {
    if (g >= ns) return ne;
    const uint64_t r = row_of(g);
    return ent0[r] + (g - seg0[r]) * kSegMax;
  }
  // end of the chunk that starts at segment a < ns: the most segments (at
  // most sc) whose entries (at most mc >= kSegMax) fit
  uint64_t chunk_end(uint64_t a, uint64_t mc, uint64_t sc) const {
    uint64_t lo = a + 1, hi = std::min(ns, a + sc);
    const uint64_t ea = entry_of(a);
    while (lo < hi) {
      const uint64_t mid = lo + (hi - lo + 1) / 2;
      if (entry_of(mid) - ea <= mc) lo = mid; else hi = mid - 1;
    }
    return lo;
  }

  // Packs segments [a, b) into the staging arrays: node (b - a), off
  // (b - a + 1, chunk-relative), col / wt (the chunk's entries; wt only for
  // a weighted G) and fold.  Returns the number of folds, or -1 if more
  // than fold_cap were needed.
  int64_t pack(HostPool& pool, const HostGraph& G, uint64_t a, uint64_t b, uint32_t* node,
               uint64_t* off, uint32_t* col, uint32_t* wt, StreamFold* fold,
               uint64_t fold_cap) const {
    const unsigned T = pool.size();
    const uint64_t ea = entry_of(a), eb = entry_of(b), len = eb - ea;
    const bool weighted = G.wt != nullptr;
    // first segment in [a, b] that starts at or after packed entry e
    auto seg_at = [&](uint64_t e) {
      uint64_t l = a, h = b;
      while (l < h) {
        const uint64_t m = l + (h - l) / 2;
        if (entry_of(m) < e) l = m + 1; else h = m;
      }
      return l;
    };
    std::vector<std::vector<StreamFold>> tf(T);
    // thread t packs the segments that start in its share of the entries
    pool.run([&](unsigned t) {
      std::vector<StreamFold>& fl = tf[t];
      const uint64_t ga = t == 0 ? a : seg_at(ea + len * t / T);
      const uint64_t gb = t + 1 == T ? b : seg_at(ea + len * (t + 1) / T);
      if (ga >= gb) return;
      uint64_t r = row_of(ga);
      uint64_t run_src = 0, run_dst = 0, run_len = 0;
      auto flush = [&] {
        if (!run_len) return;
        memcpy(col + run_dst, G.col + run_src, 4 * run_len);
        if (weighted) memcpy(wt + run_dst, G.wt + run_src, 4 * run_len);
        run_len = 0;
      };
      for (uint64_t g = ga; g < gb; ++g) {
        while (seg0[r + 1] <= g) ++r;
        const uint64_t j = g - seg0[r], nsr = seg0[r + 1] - seg0[r];
        const uint64_t rlen = ent0[r + 1] - ent0[r];
        const uint64_t pb = j * kSegMax, pl = std::min<uint64_t>(kSegMax, rlen - pb);
        const uint64_t dst = ent0[r] + pb - ea;
        const uint64_t src = G.rp(rows[r]) + pb;
        node[g - a] = rows[r] | (nsr > 1 ? kSegPartial : 0u);
        off[g - a] = dst;
        if (run_len && run_src + run_len == src && run_dst + run_len == dst) {
          run_len += pl;
        } else {
          flush();
          run_src = src;
          run_dst = dst;
          run_len = pl;
        }
        if (nsr > 1 && (j == 0 || g == a))
          fl.push_back(StreamFold{(uint32_t)(g - a), (uint32_t)(std::min(seg0[r + 1], b) - g),
                                  rows[r], j > 0 ? 1u : 0u});
      }
      flush();
    });
    off[b - a] = len;
    uint64_t nf = 0;
    for (unsigned t = 0; t < T; ++t) nf += tf[t].size();
    if (nf > fold_cap) return -1;
    nf = 0;
    for (unsigned t = 0; t < T; ++t)
      for (const StreamFold& f : tf[t]) fold[nf++] = f;
    return (int64_t)nf;
  }
};

}  // namespace wl
