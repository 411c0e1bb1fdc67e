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
