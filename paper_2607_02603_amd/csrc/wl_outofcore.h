// Host drivers of the out-of-core paths, included by wl_lib.hip after the
// in-core session (Session, open_session) they build on:
//   - Algorithm 2 (Section 4.2): batched refinement with quotient
//     contraction (batched_run), the quotient graph built on the device
//     chunk by chunk with its copies in and out on threads of their own;
//   - Algorithm 1 with the image streamed from host memory (streamed_run),
//     also the exact finish of Algorithm 2;
//   - the copies between pageable host memory and the device (HostCopy).
#pragma once

// Device workspace of the refinement phase: a batch's local CSR and labels
// plus the in-core state for up to n0 rows and mb entries.
struct RefineLayout {
  uint64_t stage, rp, col, wt, lab, colors, core, total;
};
RefineLayout refine_layout(uint64_t n0, uint64_t mb) {
  RefineLayout L{};
  uint64_t o = 0;
  auto take = [&](uint64_t b) { uint64_t at = o; o = align_up(o + b); return at; };
  L.stage = take(8 * (n0 + 1));
  L.rp = take(8 * (n0 + 1));
  L.col = take(4 * mb);
  L.wt = take(4 * mb);
  L.lab = take(4 * n0);
  L.colors = take(4 * n0);
  L.core = take(make_layout(n0, mb).total);
  L.total = o;
  return L;
}

// Device workspace of the quotient phase: block of every node, representative
// flags, a chunk of rows (mq entries) and the sort state for mq keys.
// Two sets of a chunk's input arrays: the rows of the next chunk are copied
// into one while the device reduces the current chunk from the other.
struct QuotLayout {
  uint64_t blk, isrep, stage[2], rp[2], qoff[2], col[2], wt[2], core, total;
};
QuotLayout quot_layout(uint64_t n0, uint64_t mq) {
  QuotLayout L{};
  uint64_t o = 0;
  auto take = [&](uint64_t b) { uint64_t at = o; o = align_up(o + b); return at; };
  L.blk = take(4 * n0);
  L.isrep = take(n0 + 1);
  for (int i = 0; i < 2; ++i) {
    L.stage[i] = take(8 * (n0 + 1));
    L.rp[i] = take(8 * (n0 + 1));
    L.qoff[i] = take(8 * (n0 + 1));
    L.col[i] = take(4 * mq);
    L.wt[i] = take(4 * mq);
  }
  L.core = take(make_layout(mq, 0).total);
  L.total = o;
  return L;
}

// Host array owned by the library (pageable: the quotient graphs of the outer
// iterations can be far larger than the page-locked memory a process may hold).
struct HostBuf {
  std::unique_ptr<uint8_t[]> p;
  int alloc(uint64_t bytes) {
    p.reset(new (std::nothrow) uint8_t[bytes ? bytes : 8]);
    if (!p) return fail(WL_ENOMEM, "host allocation of %llu bytes failed",
                        (unsigned long long)bytes);
    return WL_OK;
  }
  template <typename T> T* as() const { return (T*)p.get(); }
};

bool page_locked(const void* ptr) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, ptr) != hipSuccess) {
    (void)hipGetLastError();  // a pageable pointer is not an error here
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

// Copies between host memory and the device on one stream.  Page-locked host
// memory is handed to the DMA engine directly.  Pageable memory goes through
// two page-locked staging buffers: host threads fill (or drain) one while the
// DMA engine moves the other.
class HostCopy {
 public:
  static constexpr uint64_t kStage = 64ull << 20;
  explicit HostCopy(hipStream_t s) : s_(s) {
    // WL_HOST_STAGING=0: copy pageable memory without the staging buffers,
    // as when page-locked memory is refused
    const char* st = getenv("WL_HOST_STAGING");
    direct_ = st && st[0] == '0';
    cpu_set_t set;
    CPU_ZERO(&set);
    unsigned t = 4;
    if (sched_getaffinity(0, sizeof(set), &set) == 0) t = (unsigned)CPU_COUNT(&set);
    threads_ = std::max(1u, std::min(t, 8u));
  }
  ~HostCopy() {
    for (int i = 0; i < 2; ++i) {
      if (ev_[i]) {
        (void)hipEventSynchronize(ev_[i]);
        (void)hipEventDestroy(ev_[i]);
      }
      if (buf_[i]) (void)hipHostFree(buf_[i]);
    }
  }
  HostCopy(const HostCopy&) = delete;
  HostCopy& operator=(const HostCopy&) = delete;

  // Enqueues the copy; the source may be reused once the call returns.
  int h2d(void* dst, const void* src, uint64_t bytes) {
    if (bytes == 0) return WL_OK;
    if (page_locked(src)) {
      HIP_TRY(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s_));
      return WL_OK;
    }
    if (!ensure()) {
      // no page-locked staging: the runtime copies from pageable memory
      HIP_TRY(hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s_));
      HIP_TRY(hipStreamSynchronize(s_));
      return WL_OK;
    }
    for (uint64_t off = 0; off < bytes; off += kStage) {
      const uint64_t len = std::min(kStage, bytes - off);
      HIP_TRY(hipEventSynchronize(ev_[cur_]));
      par_copy(buf_[cur_], (const uint8_t*)src + off, len);
      HIP_TRY(hipMemcpyAsync((uint8_t*)dst + off, buf_[cur_], len, hipMemcpyHostToDevice, s_));
      HIP_TRY(hipEventRecord(ev_[cur_], s_));
      cur_ ^= 1;
    }
    return WL_OK;
  }

  // Returns once the data is in dst (the stream's earlier work included).
  int d2h(void* dst, const void* src, uint64_t bytes) {
    if (bytes == 0) return WL_OK;
    if (page_locked(dst)) {
      HIP_TRY(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s_));
      HIP_TRY(hipStreamSynchronize(s_));
      return WL_OK;
    }
    if (!ensure()) {
      HIP_TRY(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s_));
      HIP_TRY(hipStreamSynchronize(s_));
      return WL_OK;
    }
    int prev = -1;
    uint64_t prev_off = 0, prev_len = 0;
    for (uint64_t off = 0; off < bytes; off += kStage) {
      const uint64_t len = std::min(kStage, bytes - off);
      const int b = cur_;
      HIP_TRY(hipEventSynchronize(ev_[b]));
      HIP_TRY(hipMemcpyAsync(buf_[b], (const uint8_t*)src + off, len, hipMemcpyDeviceToHost,
                             s_));
      HIP_TRY(hipEventRecord(ev_[b], s_));
      if (prev >= 0) {
        HIP_TRY(hipEventSynchronize(ev_[prev]));
        par_copy((uint8_t*)dst + prev_off, buf_[prev], prev_len);
      }
      prev = b;
      prev_off = off;
      prev_len = len;
      cur_ ^= 1;
    }
    HIP_TRY(hipEventSynchronize(ev_[prev]));
    par_copy((uint8_t*)dst + prev_off, buf_[prev], prev_len);
    return WL_OK;
  }

 private:
  // true when the two staging buffers exist; false (for good) when the
  // page-locked memory is refused, and the copies go without them
  bool ensure() {
    if (direct_) return false;
    for (int i = 0; i < 2; ++i) {
      if (buf_[i]) continue;
      if (hipHostMalloc((void**)&buf_[i], kStage, hipHostMallocDefault) != hipSuccess ||
          hipEventCreateWithFlags(&ev_[i], hipEventDisableTiming) != hipSuccess ||
          hipEventRecord(ev_[i], s_) != hipSuccess) {
        (void)hipGetLastError();
        for (int k = 0; k < 2; ++k) {
          if (ev_[k]) {
            (void)hipEventSynchronize(ev_[k]);
            (void)hipEventDestroy(ev_[k]);
            ev_[k] = nullptr;
          }
          if (buf_[k]) (void)hipHostFree(buf_[k]);
          buf_[k] = nullptr;
        }
        direct_ = true;
        return false;
      }
    }
    return true;
  }
  void par_copy(void* d, const void* src, uint64_t len) {
    const unsigned t = len >= (4ull << 20) ? threads_ : 1;
    if (t <= 1) {
      memcpy(d, src, len);
      return;
    }
    const uint64_t per = (len + t - 1) / t;
    std::vector<std::thread> th;
    try {
      for (unsigned i = 1; i < t && i * per < len; ++i)
        th.emplace_back([=] {
          memcpy((uint8_t*)d + i * per, (const uint8_t*)src + i * per,
                 std::min(per, len - i * per));
        });
    } catch (...) {
      for (auto& x : th) x.join();
      memcpy(d, src, len);
      return;
    }
    memcpy(d, src, std::min(per, len));
    for (auto& x : th) x.join();
  }

  hipStream_t s_;
  uint8_t* buf_[2] = {nullptr, nullptr};
  hipEvent_t ev_[2] = {nullptr, nullptr};
  int cur_ = 0;
  unsigned threads_ = 1;
  bool direct_ = false;
};

int copy_rows_h2d(HostCopy& hc, const HostGraph& G, uint64_t r0, uint64_t nrows,
                  uint8_t* stage, uint64_t* rp_dev, hipStream_t s) {
  if (G.rp64) {
    if (int r = hc.h2d(stage, G.rp64 + r0, 8 * (nrows + 1))) return r;
    hipLaunchKernelGGL(k_rebase_rows<uint64_t>, dim3(grid_for(nrows + 1)), dim3(kBlock), 0,
                       s, (const uint64_t*)stage, rp_dev, (uint32_t)nrows);
  } else {
    if (int r = hc.h2d(stage, G.rp32 + r0, 4 * (nrows + 1))) return r;
    hipLaunchKernelGGL(k_rebase_rows<uint32_t>, dim3(grid_for(nrows + 1)), dim3(kBlock), 0,
                       s, (const uint32_t*)stage, rp_dev, (uint32_t)nrows);
  }
  HIP_LAUNCH_CHECK();
  return WL_OK;
}

struct QuotientOut {
  std::vector<uint64_t> deg;      // entries per block
  uint32_t* col = nullptr;        // library host arrays of capacity 'cap'
  uint32_t* wt = nullptr;
  uint64_t m = 0, cap = 0;
};

// Device buffers of one quotient chunk: the chunk's rows (rebased row
// pointers, key offsets, columns, weights); after the keys are built the
// column and weight arrays receive the distinct entries and the offsets the
// per-block entry counts.
struct QuotDev {
  uint64_t* rp;
  uint64_t* qoff;
  uint32_t* col;
  uint32_t* wt;
  uint32_t* deg() const { return (uint32_t*)qoff; }
};

// Sorts and reduces the 'nkeys' keys of one chunk on the device.  Whole rows:
// the distinct (target, weight) entries are appended to Q in key order and
// the entry counts of the chunk's 'nreps' blocks (ids bfirst ...) added to
// Q.deg; they may not reach past 'write_end' (the end of the chunk's rows
// when Q overwrites the graph it is built from).  A row processed in pieces:
// the entries go to 'spill' with 64-bit weights, merged by the caller.
int quotient_chunk(Session& S, HostCopy& hc, const QuotDev& D, uint64_t nkeys,
                   uint64_t nreps, uint32_t bfirst, uint64_t write_end, QuotientOut& Q,
                   std::vector<std::pair<uint32_t, uint64_t>>* spill,
                   std::vector<uint64_t>& hkey, std::vector<uint64_t>& hw,
                   std::vector<uint32_t>& hdeg, const std::vector<uint32_t>* seg = nullptr,
                   double* tm = nullptr, uint64_t* nd_out = nullptr) {
  // tm (diagnostics): adds the ms until the device's part is done, then the
  // ms of the copies out
  using clk = std::chrono::steady_clock;
  clk::time_point t0 = clk::now();
  // seg: key offsets of the chunk's non-empty rows and nkeys (one segment
  // each), or none (one segment)
  const uint64_t nseg = seg ? seg->size() - 1 : 0;
  if (nseg) {
    if (nseg > nkeys) return fail(WL_EINVAL, "more row segments than keys");
    if (int r = hc.h2d(S.ctx.cstart, seg->data(), 4 * (nseg + 1))) return r;
    S.host.k = (uint32_t)nseg;
  }
  hipLaunchKernelGGL(k_q_begin, dim3(grid_for(std::max(nkeys, nreps), kBlock, 4096)),
                     dim3(kBlock), 0, S.s, S.ctx, (uint32_t)nkeys, D.deg(), (uint32_t)nreps,
                     (uint32_t)nseg);
  HIP_LAUNCH_CHECK();
  if (int r = S.segmented_sort()) return r;
  hipLaunchKernelGGL(k_q_reduce, dim3(grid_for(nkeys, kBlock, 4096)), dim3(kBlock), 0, S.s,
                     S.ctx, (uint32_t)nkeys);
  HIP_LAUNCH_CHECK();
  if (spill) {
    if (int r = S.pull()) return r;
    const uint32_t nd = S.host.k_new;
    hkey.resize(nd);
    hw.resize(nd);
    if (int r = hc.d2h(hkey.data(), S.ctx.z, 8ull * nd)) return r;
    if (int r = hc.d2h(hw.data(), S.ctx.x, 8ull * nd)) return r;
    const uint64_t mask = (1ull << kQShift) - 1;
    for (uint32_t d = 0; d < nd; ++d) spill->push_back({(uint32_t)(hkey[d] & mask), hw[d]});
    return WL_OK;
  }
  hipLaunchKernelGGL(k_q_emit, dim3(grid_for(nkeys, kBlock, 4096)), dim3(kBlock), 0, S.s,
                     S.ctx, (uint32_t)nkeys, D.col, D.wt, D.deg());
  HIP_LAUNCH_CHECK();
  if (int r = S.pull()) return r;
  if (tm) {
    tm[0] += std::chrono::duration<double, std::milli>(clk::now() - t0).count();
    t0 = clk::now();
  }
  if (S.host.err & kErrQuotientWeight)
    return fail(WL_EOVERFLOW, "a quotient weight exceeds 2^32 - 1");
  const uint32_t nd = S.host.k_new;
  if (nd_out) {
    // the caller copies the chunk's entries out (quotient_chunk_out)
    *nd_out = nd;
    return WL_OK;
  }
  if (Q.m + nd > std::min(Q.cap, write_end))
    return fail(WL_EINVAL, "quotient larger than expected");
  if (int r = hc.d2h(Q.col + Q.m, D.col, 4ull * nd)) return r;
  if (int r = hc.d2h(Q.wt + Q.m, D.wt, 4ull * nd)) return r;
  hdeg.resize(nreps);
  if (int r = hc.d2h(hdeg.data(), D.deg(), 4ull * nreps)) return r;
  for (uint64_t b = 0; b < nreps; ++b) Q.deg[bfirst + b] += hdeg[b];
  Q.m += nd;
  if (tm) tm[1] += std::chrono::duration<double, std::milli>(clk::now() - t0).count();
  return WL_OK;
}


// The copies out of a reduced chunk (its nd distinct entries and the entry
// counts of its nreps blocks, ids bfirst ...), appended to Q.
int quotient_chunk_out(HostCopy& hc, const QuotDev& D, uint64_t nd, uint64_t nreps,
                       uint32_t bfirst, uint64_t write_end, QuotientOut& Q,
                       std::vector<uint32_t>& hdeg) {
  if (Q.m + nd > std::min(Q.cap, write_end))
    return fail(WL_EINVAL, "quotient larger than expected");
  if (int r = hc.d2h(Q.col + Q.m, D.col, 4ull * nd)) return r;
  if (int r = hc.d2h(Q.wt + Q.m, D.wt, 4ull * nd)) return r;
  hdeg.resize(nreps);
  if (int r = hc.d2h(hdeg.data(), D.deg(), 4ull * nreps)) return r;
  for (uint64_t b = 0; b < nreps; ++b) Q.deg[bfirst + b] += hdeg[b];
  Q.m += nd;
  return WL_OK;
}

// ---------------------------------------------------------------------------
// Algorithm 1 with the entries in host memory: the image of every round is
// streamed through the device chunk by chunk (wl_stream.h); the node state
// and the relabel stay on the device.
// ---------------------------------------------------------------------------


// Page-locked host memory owned by the library.
struct PinnedBuf {
  uint8_t* p = nullptr;
  ~PinnedBuf() { release(); }
  void release() {
    if (p) (void)hipHostFree(p);
    p = nullptr;
  }
  // false when the allocation is refused (page-locked memory is limited)
  bool try_alloc(uint64_t bytes) {
    release();
    if (hipHostMalloc((void**)&p, bytes ? bytes : 8, hipHostMallocDefault) != hipSuccess) {
      p = nullptr;
      (void)hipGetLastError();
      return false;
    }
    return true;
  }
};

constexpr uint64_t kStreamMaxChunk = 64ull << 20;  // entries per chunk
constexpr uint64_t kStreamMinStage = 1ull << 16;   // smallest staged chunk (entries)


// One chunk's arrays (device slot, or host staging without 'part').
struct StreamSlot {
  uint64_t node, off, col, wt, part, fold, total;
};
StreamSlot stream_slot(uint64_t mc, bool weighted, bool device) {
  StreamSlot L{};
  uint64_t o = 0;
  auto take = [&](uint64_t b) { uint64_t at = o; o = align_up(o + b); return at; };
  const uint64_t sc = stream_segs(mc);
  L.node = take(4 * sc);
  L.off = take(8 * (sc + 1));
  L.col = take(4 * mc);
  L.wt = take(weighted ? 4 * mc : 0);
  L.part = take(device ? 8 * sc : 0);
  L.fold = take(16 * stream_folds(mc));
  L.total = o;
  return L;
}

struct StreamLayout {
  uint64_t core, core_bytes, colors, slot[2], total;
  StreamSlot sl;
};
StreamLayout stream_layout(uint64_t n, uint64_t mc, bool weighted) {
  StreamLayout L{};
  uint64_t o = 0;
  auto take = [&](uint64_t b) { uint64_t at = o; o = align_up(o + b); return at; };
  L.core_bytes = make_layout(n, 0, false).total;
  L.core = take(L.core_bytes);
  L.colors = take(4 * n);
  L.sl = stream_slot(mc, weighted, true);
  L.slot[0] = take(L.sl.total);
  L.slot[1] = take(L.sl.total);
  L.total = o;
  return L;
}

uint64_t stream_chunk_cap(const HostGraph& G) {
  return std::min<uint64_t>(kStreamMaxChunk, std::max<uint64_t>(G.m, 1));
}

// Events and the copy stream of the streamed rounds.
struct StreamRes {
  hipStream_t cs = nullptr;
  hipEvent_t copied[2] = {nullptr, nullptr}, computed[2] = {nullptr, nullptr};
  ~StreamRes() {
    if (cs) (void)hipStreamSynchronize(cs);
    for (int i = 0; i < 2; ++i) {
      if (copied[i]) (void)hipEventDestroy(copied[i]);
      if (computed[i]) (void)hipEventDestroy(computed[i]);
    }
    if (cs) (void)hipStreamDestroy(cs);
  }
};

// Algorithm 1 on the host graph G from its labels (or the trivial
// partition).  Colours (raw rank ids, as in the in-core path) to color_host;
// *done_out: 1 stable, 2 round cap reached.
int streamed_run(const HostGraph& G, const uint32_t* labels, uint64_t seed,
                 uint32_t max_rounds, uint8_t* W, uint64_t ws_bytes, hipStream_t s,
                 uint32_t* color_host, uint32_t* k_out, uint32_t* rounds_out, int* done_out) {
  const uint64_t n = G.n;
  const bool weighted = G.wt != nullptr;
  const char* trs = getenv("WL_TRACE_STREAMED");
  const bool trace = trs && trs[0] == '1';
  using clk = std::chrono::steady_clock;
  auto ms_since = [](clk::time_point t) {
    return std::chrono::duration<double, std::milli>(clk::now() - t).count();
  };
  const clk::time_point t_call = clk::now();
  const uint64_t mc = largest_fitting(
      [&](uint64_t c) { return stream_layout(n, c, weighted).total; }, ws_bytes,
      stream_chunk_cap(G));
  if (mc < std::min<uint64_t>(kSegMax, std::max<uint64_t>(G.m, 1)))
    return fail(WL_EBUDGET, "workspace of %llu bytes holds no chunk of %u entries",
                (unsigned long long)ws_bytes, kSegMax);
  const StreamLayout SL = stream_layout(n, mc, weighted);
  uint32_t* colors_dev = (uint32_t*)(W + SL.colors);
  wl_csr vg{};
  vg.n = n;
  Session S;
  if (int r = open_session(S, &vg, colors_dev, W + SL.core, SL.core_bytes, s, false)) return r;
  const uint32_t cap = max_rounds ? max_rounds : (uint32_t)std::min<uint64_t>(n + 1, 0xFFFFFFFFull);
  if (int r = S.init_state(seed, 1, 0, cap, 1)) return r;
  if (int r = S.stats_begin()) return r;

  HostPool pool;
  const unsigned T = pool.size();
  // page-locked staging for two chunks; the chunk shrinks when that much
  // page-locked memory is refused (the device slots keep their size)
  PinnedBuf stage[2];
  uint64_t mcs = mc;
  for (;;) {
    const uint64_t bytes = stream_slot(mcs, weighted, false).total;
    if (stage[0].try_alloc(bytes) && stage[1].try_alloc(bytes)) break;
    stage[0].release();
    stage[1].release();
    if (mcs <= std::min(kStreamMinStage, mc))
      return fail(WL_ENOMEM, "no page-locked staging of %llu bytes",
                  (unsigned long long)bytes);
    mcs = std::max(std::min(kStreamMinStage, mc), mcs / 2);
  }
  const StreamSlot HS = stream_slot(mcs, weighted, false);
  const uint64_t sc = stream_segs(mcs);
  if (trace)
    fprintf(stderr, "[wl streamed] n=%llu m=%llu chunk=%llu staged=%llu set-up %.1f ms\n",
            (unsigned long long)n, (unsigned long long)G.m, (unsigned long long)mc,
            (unsigned long long)mcs, ms_since(t_call));
  std::vector<uint8_t> act_h;
  StreamRes R;
  HIP_TRY(hipStreamCreateWithFlags(&R.cs, hipStreamNonBlocking));
  for (int i = 0; i < 2; ++i) {
    HIP_TRY(hipEventCreateWithFlags(&R.copied[i], hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&R.computed[i], hipEventDisableTiming));
    HIP_TRY(hipEventRecord(R.copied[i], R.cs));
    HIP_TRY(hipEventRecord(R.computed[i], s));
  }
  HostCopy hc(s);

  const uint32_t gn = grid_for(n, kBlock, 4096);
  hipLaunchKernelGGL(k_iota_zero, dim3(gn), dim3(kBlock), 0, s, S.ctx);
  HIP_LAUNCH_CHECK();
  if (labels) {
    uint32_t* lab_dev = (uint32_t*)S.ctx.x;
    if (int r = hc.h2d(lab_dev, labels, 4 * n)) return r;
    hipLaunchKernelGGL(k_labels_to_z, dim3(gn), dim3(kBlock), 0, s, S.ctx, lab_dev);
    HIP_LAUNCH_CHECK();
    if (int r = S.relabel(0)) return r;
  }

  StreamPlan plan;
  // Once all chunks of a round fit in the workspace beyond its layout, they
  // are copied there instead of to the two slots and kept: the rows a later
  // round needs are among them (a class never grows back), and the image of
  // a row that is no longer needed is not used.
  bool resident = false;
  std::vector<StreamChunk> res_chunks;
  const uint64_t keep_begin = align_up(SL.total);
  const uint64_t keep_bytes = ws_bytes > keep_begin ? ws_bytes - keep_begin : 0;
  // a kept chunk's arrays, packed: node, off, col, wt, part, fold
  auto kept_layout = [&](uint64_t nseg, uint64_t len, uint64_t nf, uint64_t o[6]) {
    uint64_t at = 0;
    const uint64_t sz[6] = {4 * nseg, 8 * (nseg + 1), 4 * len, weighted ? 4 * len : 0, 8 * nseg,
                            16 * nf};
    for (int i = 0; i < 6; ++i) {
      o[i] = at;
      at = align_up(at + sz[i]);
    }
    return at;
  };
  auto launch_chunk = [&](const StreamChunk& ch) -> int {
    const uint32_t gs = grid_for(ch.nseg, kBlock / kWave, 16384);
    if (weighted)
      hipLaunchKernelGGL(k_stream_seg<true>, dim3(gs), dim3(kBlock), 0, s, S.ctx, ch);
    else
      hipLaunchKernelGGL(k_stream_seg<false>, dim3(gs), dim3(kBlock), 0, s, S.ctx, ch);
    if (ch.nfold)
      hipLaunchKernelGGL(k_stream_fold, dim3(grid_for(ch.nfold, kBlock, 1024)), dim3(kBlock), 0,
                         s, S.ctx, ch);
    HIP_LAUNCH_CHECK();
    return WL_OK;
  };

  while (!S.host.done) {
    const clk::time_point t_round = clk::now();
    double pack_ms = 0, wait_ms = 0, act_ms = 0, plan_ms = 0, relabel_ms = 0;
    uint64_t chunks = 0;
    hipLaunchKernelGGL(k_round_begin, dim3(1), dim3(1), 0, s, S.ctx);
    HIP_LAUNCH_CHECK();
    bool uniform = S.host.k == 1 && !weighted;
    if (uniform) {
      // z_i = deg_i * w: the degrees only, computed by host threads straight
      // into the two page-locked staging buffers and copied chunk by chunk
      uint32_t* deg_dev = (uint32_t*)S.ctx.keys_tmp;
      const uint64_t per = HS.total / 4;  // degrees per staging buffer
      std::vector<uint8_t> big(T, 0);
      int slot = 0;
      // the copies overwrite scratch that earlier work on s may still use
      HIP_TRY(hipEventRecord(R.computed[0], s));
      HIP_TRY(hipStreamWaitEvent(R.cs, R.computed[0], 0));
      for (uint64_t r0 = 0; r0 < n; r0 += per) {
        const uint64_t nr = std::min(per, n - r0);
        HIP_TRY(hipEventSynchronize(R.copied[slot]));
        uint32_t* deg = (uint32_t*)stage[slot].p;
        pool.run([&](unsigned t) {
          for (uint64_t i = nr * t / T; i < nr * (t + 1) / T; ++i) {
            const uint64_t d = G.rp(r0 + i + 1) - G.rp(r0 + i);
            if (d > 0xFFFFFFFFull) big[t] = 1;
            deg[i] = (uint32_t)d;
          }
        });
        HIP_TRY(hipMemcpyAsync(deg_dev + r0, deg, 4 * nr, hipMemcpyHostToDevice, R.cs));
        HIP_TRY(hipEventRecord(R.copied[slot], R.cs));
        slot ^= 1;
      }
      HIP_TRY(hipStreamWaitEvent(s, R.copied[slot ^ 1], 0));
      HIP_TRY(hipStreamWaitEvent(s, R.copied[slot], 0));
      for (unsigned t = 0; t < T; ++t) uniform = uniform && !big[t];
      if (uniform) {
        hipLaunchKernelGGL(k_stream_uniform, dim3(gn), dim3(kBlock), 0, s, S.ctx, deg_dev);
        HIP_LAUNCH_CHECK();
      }
    }
    if (!uniform) {
      act_h.resize(n);
      hipLaunchKernelGGL(k_zero_u64, dim3(grid_for(n, kBlock, 4096)), dim3(kBlock), 0, s,
                         S.ctx.z, n);
      hipLaunchKernelGGL(k_gather_prep, dim3(gn), dim3(kBlock), 0, s, S.ctx, -1);
      HIP_LAUNCH_CHECK();
    }
    if (!uniform && resident) {
      for (const StreamChunk& ch : res_chunks)
        if (int r = launch_chunk(ch)) return r;
    } else if (!uniform) {
      clk::time_point t0 = clk::now();
      if (int r = hc.d2h(act_h.data(), S.ctx.act, n)) return r;
      act_ms = ms_since(t0);
      t0 = clk::now();
      if (!plan.build(pool, G, act_h.data()))
        return fail(WL_ENOMEM, "host arrays for the plan of %llu rows",
                    (unsigned long long)n);
      plan_ms = ms_since(t0);
      // keep this round's chunks if they all fit (a bound of their bytes)
      uint64_t nchunks = 0;
      for (uint64_t a = 0; a < plan.ns; a = plan.chunk_end(a, mcs, sc)) ++nchunks;
      const uint64_t bound = 20 * plan.ns + (weighted ? 8 : 4) * plan.ne +
                             nchunks * (8 + 16 * stream_folds(mcs) + 6 * kAlign);
      const bool keep = plan.ns > 0 && bound <= keep_bytes;
      uint64_t keep_off = keep_begin;
      uint64_t a = 0;
      int slot = 0;
      while (a < plan.ns) {
        const uint64_t b = plan.chunk_end(a, mcs, sc);
        const uint64_t len = plan.entry_of(b) - plan.entry_of(a), nseg = b - a;
        clk::time_point t0 = clk::now();
        HIP_TRY(hipEventSynchronize(R.copied[slot]));
        wait_ms += ms_since(t0);
        t0 = clk::now();
        ++chunks;
        uint8_t* H = stage[slot].p;
        uint32_t* hnode = (uint32_t*)(H + HS.node);
        uint64_t* hoff = (uint64_t*)(H + HS.off);
        uint32_t* hcol = (uint32_t*)(H + HS.col);
        uint32_t* hwt = (uint32_t*)(H + HS.wt);
        StreamFold* hfold = (StreamFold*)(H + HS.fold);
        const int64_t nfs = plan.pack(pool, G, a, b, hnode, hoff, hcol, weighted ? hwt : nullptr,
                                      hfold, stream_folds(mcs));
        if (nfs < 0) return fail(WL_EINVAL, "chunk plan exceeds its fold table");
        pack_ms += ms_since(t0);
        const uint64_t nf = (uint64_t)nfs;
        uint8_t* D;
        uint64_t o[6] = {SL.sl.node, SL.sl.off, SL.sl.col, SL.sl.wt, SL.sl.part, SL.sl.fold};
        if (keep) {
          D = W + keep_off;
          const uint64_t tot = kept_layout(nseg, len, nf, o);
          if (keep_off + tot > keep_begin + keep_bytes)
            return fail(WL_EINVAL, "kept chunks exceed their bound");
          keep_off += tot;
        } else {
          D = W + SL.slot[slot];
          HIP_TRY(hipStreamWaitEvent(R.cs, R.computed[slot], 0));
        }
        HIP_TRY(hipMemcpyAsync(D + o[0], hnode, 4 * nseg, hipMemcpyHostToDevice, R.cs));
        HIP_TRY(hipMemcpyAsync(D + o[1], hoff, 8 * (nseg + 1), hipMemcpyHostToDevice, R.cs));
        HIP_TRY(hipMemcpyAsync(D + o[2], hcol, 4 * len, hipMemcpyHostToDevice, R.cs));
        if (weighted)
          HIP_TRY(hipMemcpyAsync(D + o[3], hwt, 4 * len, hipMemcpyHostToDevice, R.cs));
        if (nf) HIP_TRY(hipMemcpyAsync(D + o[5], hfold, 16 * nf, hipMemcpyHostToDevice, R.cs));
        HIP_TRY(hipEventRecord(R.copied[slot], R.cs));
        HIP_TRY(hipStreamWaitEvent(s, R.copied[slot], 0));
        StreamChunk ch;
        ch.node = (const uint32_t*)(D + o[0]);
        ch.off = (const uint64_t*)(D + o[1]);
        ch.col = (const uint32_t*)(D + o[2]);
        ch.wt = weighted ? (const uint32_t*)(D + o[3]) : nullptr;
        ch.part = (uint64_t*)(D + o[4]);
        ch.fold = (const StreamFold*)(D + o[5]);
        ch.nseg = (uint32_t)nseg;
        ch.nfold = (uint32_t)nf;
        if (int r = launch_chunk(ch)) return r;
        HIP_TRY(hipEventRecord(R.computed[slot], s));
        if (keep) res_chunks.push_back(ch);
        a = b;
        slot ^= 1;
      }
      resident = keep;
    }
    if (trace) {
      HIP_TRY(hipStreamSynchronize(s));
      const clk::time_point t0 = clk::now();
      if (int r = S.relabel(1)) return r;
      relabel_ms = ms_since(t0);
    } else if (int r = S.relabel(1)) {
      return r;
    }
    if (trace)
      fprintf(stderr, "[wl streamed] round %u: %s rows %llu entries %llu chunks %llu, "
              "act %.1f ms, plan %.1f ms, packing %.1f ms, waiting for copies %.1f ms, "
              "relabel %.1f ms, round %.1f ms, colours %u\n",
              S.host.round, uniform ? "degrees," : (resident && !chunks ? "resident chunk," : ""),
              uniform ? 0ull : (unsigned long long)plan.nr,
              uniform ? 0ull : (unsigned long long)plan.ne, (unsigned long long)chunks, act_ms,
              plan_ms, pack_ms, wait_ms, relabel_ms, ms_since(t_round), S.host.k);
  }
  if (int r = S.stats_end()) return r;
  if (int r = hc.d2h(color_host, colors_dev, 4 * n)) return r;
  if (trace) fprintf(stderr, "[wl streamed] call %.1f ms\n", ms_since(t_call));
  *k_out = S.host.k;
  *rounds_out = S.host.round;
  *done_out = (int)S.host.done;
  return WL_OK;
}

int batched_run(const wl_csr* g, const uint32_t* init_host, uint64_t seed,
                uint64_t max_batch, uint32_t options, uint32_t* color_out, uint32_t* k_out,
                uint32_t* rounds_out, uint32_t* outer_out, int* coarsest_out,
                void* ws, uint64_t ws_bytes, hipStream_t s) {
  const uint64_t n0 = g->n;
  const bool exact = (options & WL_BATCHED_EXACT) != 0;
  const bool early = (options & WL_BATCHED_EARLY_STOP) != 0;
  uint8_t* W = (uint8_t*)ws;
  const char* tr = getenv("WL_TRACE_BATCHED");
  const bool trace = tr && tr[0] == '1';
  using clk = std::chrono::steady_clock;
  auto ms_since = [](clk::time_point t) {
    return std::chrono::duration<double, std::milli>(clk::now() - t).count();
  };
  clk::time_point t_phase = clk::now();

  HostGraph G;
  G.n = n0;
  G.m = g->nnz;
  G.rp32 = g->row_ptr32;
  G.rp64 = g->row_ptr64;
  G.col = g->col_idx;
  G.wt = g->weight;
  std::vector<uint32_t> labels;  // labels of G_t's nodes (raw), empty = none
  if (init_host) labels.assign(init_host, init_host + n0);
  std::vector<uint32_t> map0(n0);
  for (uint64_t i = 0; i < n0; ++i) map0[i] = (uint32_t)i;
  HostBuf qrp_buf, qcol_buf, qwt_buf;  // current quotient (G_t, t >= 1)
  HostBuf nrp_buf, ncol_buf, nwt_buf;  // G_1 under construction, new row pointers
  HostCopy hc(s);
  // copy streams and staging of the quotient pipeline (kept over the outer
  // iterations; page-locked memory is not given back and taken again)
  struct QStreams {
    hipStream_t in = nullptr, out = nullptr;
    ~QStreams() {
      for (hipStream_t x : {in, out})
        if (x) {
          (void)hipStreamSynchronize(x);
          (void)hipStreamDestroy(x);
        }
    }
  } qstr;
  HIP_TRY(hipStreamCreateWithFlags(&qstr.in, hipStreamNonBlocking));
  HIP_TRY(hipStreamCreateWithFlags(&qstr.out, hipStreamNonBlocking));
  HostCopy hc_in(qstr.in), hc_out(qstr.out);
  uint64_t rounds = 0;
  uint32_t outer = 0;
  std::vector<uint32_t> key, loc;
  RawBuf<uint32_t> blk, mapk;
  RawBuf<uint8_t> isrep;
  HostPool pool;
  std::vector<uint64_t> hkey, hw;
  std::vector<uint32_t> hdeg;
  std::vector<uint64_t> piece_rp(3);

  // batch cap for graph G: the caller's, or the largest whose batches fit
  auto plan_batches = [&](const HostGraph& Gp, uint64_t* mb_out,
                          std::vector<uint64_t>* starts_out) -> int {
    const uint64_t mall = std::max<uint64_t>(Gp.m, 1);  // a cap >= nnz is one batch
    if (max_batch) {
      *mb_out = std::min(max_batch, mall);
    } else {
      const uint64_t cap = fit_batch_cap(Gp, ws_bytes, [](uint64_t rows, uint64_t c) {
        return refine_layout(rows, c).total;
      });
      if (cap == 0)
        return fail(WL_EBUDGET, "workspace of %llu bytes holds no batch",
                    (unsigned long long)ws_bytes);
      *mb_out = cap;
    }
    *starts_out = cut_batches(Gp, *mb_out);
    return WL_OK;
  };
  // Algorithm 1 on Gf with its entries streamed from host memory; the
  // result, lifted through map0, is the final colouring
  auto finish_exact = [&](const HostGraph& Gf) -> int {
    std::vector<uint32_t> col_f(Gf.n);
    uint32_t kf = 0, rf = 0;
    int done = 0;
    if (int r = streamed_run(Gf, labels.empty() ? nullptr : labels.data(), seed, 0, W,
                             ws_bytes, s, col_f.data(), &kf, &rf, &done))
      return r;
    if (done == 2) return fail(WL_EMAXROUNDS, "streamed refinement did not stabilise");
    rounds += rf;
    if (trace)
      fprintf(stderr, "[wl batched] exact finish on n=%llu m=%llu: colours %u rounds %u\n",
              (unsigned long long)Gf.n, (unsigned long long)Gf.m, kf, rf);
    canonical_colours(map0, col_f.data(), Gf.n, color_out, k_out);
    *rounds_out = (uint32_t)std::min<uint64_t>(rounds, 0xFFFFFFFFull);
    *outer_out = outer;
    *coarsest_out = 1;
    return WL_OK;
  };
  uint64_t mb = 0;
  std::vector<uint64_t> starts;
  if (int r = plan_batches(G, &mb, &starts)) return r;

  for (uint64_t t = 0;; ++t) {
    const uint64_t n = G.n;
    const uint64_t nb = starts.size() - 1;
    const uint64_t rows_cap = max_inner_rows(G, starts);
    const RefineLayout RL = refine_layout(rows_cap, mb);
    if (RL.total > ws_bytes)
      return fail(WL_EBUDGET, "a batch of %llu entries and %llu rows needs %llu bytes, "
                  "the workspace has %llu", (unsigned long long)mb,
                  (unsigned long long)rows_cap, (unsigned long long)RL.total,
                  (unsigned long long)ws_bytes);
    const uint64_t mq = largest_fitting(
        [&](uint64_t q) { return quot_layout(n, q).total; }, ws_bytes, (1ull << 31) - 1);
    if (mq == 0) return fail(WL_EBUDGET, "workspace too small for the quotient phase");
    if (trace)
      fprintf(stderr, "[wl batched] t=%llu n=%llu m=%llu cap=%llu batches=%llu rows_cap=%llu "
              "quotient_chunk=%llu (%.1f ms since the last line)\n", (unsigned long long)t,
              (unsigned long long)n, (unsigned long long)G.m, (unsigned long long)mb,
              (unsigned long long)nb, (unsigned long long)rows_cap, (unsigned long long)mq,
              ms_since(t_phase));
    if (trace) t_phase = clk::now();
    // ---- refinement of every batch (Eq. batch-init), merge keys (Eq. merge)
    key.resize(n);
    pool.run([&](unsigned th) {
      std::fill(key.begin() + n * th / pool.size(), key.begin() + n * (th + 1) / pool.size(),
                kNoKey);
    });
    uint64_t base = 0;
    for (uint64_t b = 0; b < nb; ++b) {
      uint64_t r_lo, r_hi;
      inner_rows(G, starts, b, &r_lo, &r_hi);
      if (r_hi <= r_lo) {
        // no inner node: every node is a frozen singleton, Algorithm 1 stops
        // after the one round that confirms it
        rounds += 1;
        continue;
      }
      const uint64_t nl = r_hi - r_lo, e0 = G.rp(r_lo), ml = G.rp(r_hi) - e0;
      uint64_t* rp_dev = (uint64_t*)(W + RL.rp);
      uint32_t* col_dev = (uint32_t*)(W + RL.col);
      uint32_t* wt_dev = G.wt ? (uint32_t*)(W + RL.wt) : nullptr;
      uint32_t* lab_dev = labels.empty() ? nullptr : (uint32_t*)(W + RL.lab);
      uint32_t* colors_dev = (uint32_t*)(W + RL.colors);
      if (int r = copy_rows_h2d(hc, G, r_lo, nl, W + RL.stage, rp_dev, s)) return r;
      if (int r = hc.h2d(col_dev, G.col + e0, 4 * ml)) return r;
      if (wt_dev)
        if (int r = hc.h2d(wt_dev, G.wt + e0, 4 * ml)) return r;
      if (lab_dev)
        if (int r = hc.h2d(lab_dev, labels.data() + r_lo, 4 * nl)) return r;
      wl_csr lg{};
      lg.n = nl;
      lg.nnz = ml;
      lg.row_ptr64 = rp_dev;
      lg.col_idx = col_dev;
      lg.weight = wt_dev;
      Session S;
      if (int r = open_session(S, &lg, colors_dev, W + RL.core, RL.total - RL.core, s))
        return r;
      S.ctx.batch = 1;
      S.ctx.ext_lo = (uint32_t)r_lo;
      const uint64_t sb_seed = seed + ((t << 32) + b + 1) * 0x9E3779B97F4A7C15ull;
      uint64_t z = sb_seed;  // mix(seed + (2^32 t + b + 1) g)
      z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
      z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
      z ^= z >> 31;
      if (int r = S.init_state(z, 1, 0, (uint32_t)std::min<uint64_t>(nl + 1, 0xFFFFFFFFull), 1))
        return r;
      if (int r = S.run_rsc(lab_dev)) return r;
      if (S.host.done == 2) return fail(WL_EMAXROUNDS, "batch refinement did not stabilise");
      rounds += S.host.round;
      if (trace)
        fprintf(stderr, "[wl batched]   batch %llu rows [%llu, %llu) entries %llu colours %u "
              "rounds %u (%.1f ms since the last line)\n",
                (unsigned long long)b, (unsigned long long)r_lo, (unsigned long long)r_hi,
                (unsigned long long)ml, S.host.k, S.host.round, ms_since(t_phase));
    if (trace) t_phase = clk::now();
      loc.resize(nl);
      if (int r = hc.d2h(loc.data(), colors_dev, 4 * nl)) return r;
      for (uint64_t i = 0; i < nl; ++i) key[r_lo + i] = (uint32_t)(base + loc[i]);
      base += S.host.k;
    }
    // ---- merged partition: first-occurrence ids; boundary nodes singletons
    if (!mapk.reserve(base) || !blk.reserve(n) || !isrep.reserve(n))
      return fail(WL_ENOMEM, "host arrays of the merged partition (%llu nodes)",
                  (unsigned long long)n);
    const uint64_t nq = merge_blocks(pool, key.data(), n, base, mapk.p.get(), blk.p.get(),
                                     isrep.p.get());
    ++outer;
    if (trace)
      fprintf(stderr, "[wl batched] t=%llu merged blocks=%llu rounds so far=%llu (merge %.1f ms)\n",
              (unsigned long long)t, (unsigned long long)nq, (unsigned long long)rounds,
              ms_since(t_phase));
    if (trace) t_phase = clk::now();
    // fixed point with several batches: the exact finish runs on G_t itself
    if (nb > 1 && nq == n && exact) return finish_exact(G);
    pool.run([&](unsigned th) {
      for (uint64_t v = n0 * th / pool.size(); v < n0 * (th + 1) / pool.size(); ++v)
        map0[v] = blk[map0[v]];
    });
    if (nb == 1 || nq == n) {
      *coarsest_out = (nb == 1) ? 1 : 0;
      break;
    }
    // ---- quotient graph (Definition "Quotient Graph"), on the device
    std::vector<uint64_t> qcap_t(pool.size(), 0);
    pool.run([&](unsigned th) {
      uint64_t c = 0;
      for (uint64_t i = n * th / pool.size(); i < n * (th + 1) / pool.size(); ++i)
        if (isrep[i]) c += G.rp(i + 1) - G.rp(i);
      qcap_t[th] = c;
    });
    uint64_t qcap = 0;
    for (uint64_t c : qcap_t) qcap += c;
    QuotientOut Q;
    Q.deg.assign(nq, 0);
    const bool in_place = t > 0;
    if (in_place) {
      // G_t is the library's own: G_{t+1} overwrites it.  Block ids follow
      // their representatives' node order and a block's row is never longer
      // than its representative's, so every entry is written at or before
      // the start of the row it comes from, which has been copied by then.
      Q.col = qcol_buf.as<uint32_t>();
      Q.wt = qwt_buf.as<uint32_t>();
      Q.cap = G.m;
    } else {
      if (int r = ncol_buf.alloc(4 * qcap)) return r;
      if (int r = nwt_buf.alloc(4 * qcap)) return r;
      Q.col = ncol_buf.as<uint32_t>();
      Q.wt = nwt_buf.as<uint32_t>();
      Q.cap = qcap;
    }
    const QuotLayout QL = quot_layout(n, mq);
    uint32_t* blk_dev = (uint32_t*)(W + QL.blk);
    uint8_t* isrep_dev = W + QL.isrep;
    const QuotDev Ds[2] = {
        {(uint64_t*)(W + QL.rp[0]), (uint64_t*)(W + QL.qoff[0]), (uint32_t*)(W + QL.col[0]),
         (uint32_t*)(W + QL.wt[0])},
        {(uint64_t*)(W + QL.rp[1]), (uint64_t*)(W + QL.qoff[1]), (uint32_t*)(W + QL.col[1]),
         (uint32_t*)(W + QL.wt[1])}};
    if (int r = hc.h2d(blk_dev, blk.data(), 4 * n)) return r;
    if (int r = hc.h2d(isrep_dev, isrep.data(), n)) return r;
    // chunks: row ranges [a, bnd) of at most mq entries, or one row longer
    // than that (processed in pieces)
    const std::vector<QChunk> qch = quotient_chunks(G, mq);
    // Pipeline: a host thread prepares chunk j+1 (its key offsets, and the
    // copies of its rows into input set (j+1) & 1 on a copy stream of its
    // own) while this thread reduces chunk j from set j & 1.  A set is
    // refilled only after the chunk that used it two steps before has been
    // reduced and copied out.
    QChunkPrep qs[2];
    struct QPipe {
      std::mutex m;
      std::condition_variable cv;
      uint64_t prepared = 0, released = 0;
      bool stop = false;
      int err = WL_OK;
      std::string msg;
      hipStream_t cs = nullptr;
      hipEvent_t ready[2] = {nullptr, nullptr};
      std::thread th;
      ~QPipe() {
        {
          std::lock_guard<std::mutex> g(m);
          stop = true;
        }
        cv.notify_all();
        if (th.joinable()) th.join();
        if (cs) (void)hipStreamSynchronize(cs);
        for (auto& e : ready)
          if (e) (void)hipEventDestroy(e);
      }
    } qp;
    qp.cs = qstr.in;
    for (auto& e : qp.ready) HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    auto prefetch = [&] {
      HostCopy& hc2 = hc_in;
      for (uint64_t j = 0; j < qch.size(); ++j) {
        {
          std::unique_lock<std::mutex> g(qp.m);
          qp.cv.wait(g, [&] { return qp.stop || j < 2 || qp.released + 1 >= j; });
          if (qp.stop) return;
        }
        const QChunk& c = qch[j];
        const int st = (int)(j & 1);
        QChunkPrep& q = qs[st];
        int rc = WL_OK;
        if (c.ent <= mq) {
          const uint64_t nrows = c.bnd - c.a;
          prep_quotient_chunk(G, c, isrep.data(), blk.data(), q);
          if (q.run > 0) {
            const QuotDev& D = Ds[st];
            rc = copy_rows_h2d(hc2, G, c.a, nrows, W + QL.stage[st], D.rp, qp.cs);
            if (!rc) rc = hc2.h2d(D.qoff, q.qoff.data(), 8 * nrows);
            if (!rc) rc = hc2.h2d(D.col, G.col + c.ea, 4 * c.ent);
            if (!rc && G.wt) rc = hc2.h2d(D.wt, G.wt + c.ea, 4 * c.ent);
            if (!rc && hipEventRecord(qp.ready[st], qp.cs) != hipSuccess)
              rc = fail(WL_EHIP, "hipEventRecord failed");
          }
        }
        std::lock_guard<std::mutex> g(qp.m);
        if (rc) {
          qp.err = rc;
          qp.msg = g_err;
          qp.stop = true;
        }
        qp.prepared = j + 1;
        qp.cv.notify_all();
        if (rc) return;
      }
    };
    // a host allocation failing inside the thread ends it with WL_ENOMEM
    auto prefetch_guarded = [&] {
      try {
        prefetch();
      } catch (...) {
        std::lock_guard<std::mutex> g(qp.m);
        qp.err = WL_ENOMEM;
        qp.msg = "host allocation failed while preparing a quotient chunk";
        qp.stop = true;
        qp.cv.notify_all();
      }
    };
    try {
      qp.th = std::thread(prefetch_guarded);
    } catch (...) {
      return fail(WL_ENOMEM, "no host thread for the quotient copies");
    }
    // A second host thread copies the entries of reduced chunk j out (on a
    // stream of its own) while this thread reduces chunk j+1; it releases the
    // chunks' input sets in chunk order.
    struct QJob {
      uint64_t j, nd, nreps, write_end;
      uint32_t bfirst;
      bool copy;
    };
    struct QOut {
      std::mutex m;
      std::condition_variable cv;
      std::deque<QJob> jobs;
      uint64_t done = 0;
      bool stop = false;
      int err = WL_OK;
      std::string msg;
      hipStream_t cs = nullptr;
      std::thread th;
      ~QOut() {
        {
          std::lock_guard<std::mutex> g(m);
          stop = true;
        }
        cv.notify_all();
        if (th.joinable()) th.join();
        if (cs) (void)hipStreamSynchronize(cs);
      }
    } qo;
    qo.cs = qstr.out;
    auto drain = [&] {
      HostCopy& hc3 = hc_out;
      std::vector<uint32_t> hdeg3;
      for (;;) {
        QJob jb;
        {
          std::unique_lock<std::mutex> g(qo.m);
          qo.cv.wait(g, [&] { return qo.stop || !qo.jobs.empty(); });
          if (qo.jobs.empty()) return;
          jb = qo.jobs.front();
          qo.jobs.pop_front();
        }
        int rc = WL_OK;
        if (jb.copy)
          rc = quotient_chunk_out(hc3, Ds[jb.j & 1], jb.nd, jb.nreps, jb.bfirst, jb.write_end, Q,
                                  hdeg3);
        {
          std::lock_guard<std::mutex> g(qo.m);
          if (rc) {
            qo.err = rc;
            qo.msg = g_err;
          }
          qo.done = jb.j + 1;
          qo.cv.notify_all();
        }
        {
          // a failed copy also stops the preparation and wakes this thread's
          // partner waiting for the next chunk
          std::lock_guard<std::mutex> g(qp.m);
          qp.released = jb.j + 1;
          if (rc) {
            qp.err = rc;
            qp.msg = g_err;
            qp.stop = true;
          }
          qp.cv.notify_all();
        }
        if (rc) return;
      }
    };
    auto drain_guarded = [&] {
      try {
        drain();
      } catch (...) {
        const char* msg = "host allocation failed while copying a quotient chunk out";
        {
          std::lock_guard<std::mutex> g(qo.m);
          qo.err = WL_ENOMEM;
          qo.msg = msg;
          qo.cv.notify_all();
        }
        std::lock_guard<std::mutex> g(qp.m);
        qp.err = WL_ENOMEM;
        qp.msg = msg;
        qp.stop = true;
        qp.cv.notify_all();
      }
    };
    try {
      qo.th = std::thread(drain_guarded);
    } catch (...) {
      return fail(WL_ENOMEM, "no host thread for the quotient copies");
    }
    auto push_job = [&](const QJob& jb) {
      std::lock_guard<std::mutex> g(qo.m);
      qo.jobs.push_back(jb);
      qo.cv.notify_all();
    };
    // waits until the copies out of every chunk before j are done
    auto wait_out = [&](uint64_t j) -> int {
      std::unique_lock<std::mutex> g(qo.m);
      qo.cv.wait(g, [&] { return qo.err != WL_OK || qo.done >= j; });
      return qo.err;
    };
    double q_dev_ms = 0, q_tm[2] = {0, 0};
    uint64_t q_chunks = 0;
    for (uint64_t j = 0; j < qch.size(); ++j) {
      {
        std::unique_lock<std::mutex> g(qp.m);
        qp.cv.wait(g, [&] { return qp.err != WL_OK || qp.prepared > j; });
        if (qp.err != WL_OK) return fail(qp.err, "%s", qp.msg.c_str());
      }
      const QChunk& c = qch[j];
      const int st = (int)(j & 1);
      const QuotDev& D = Ds[st];
      const uint64_t a = c.a, ea = c.ea, ent = c.ent;
      if (ent > mq) {
        // a single row longer than the chunk: pieces, merged on the host
        // (after the copies out of the chunks before it: Q grows in order)
        if (wait_out(j)) return fail(qo.err, "%s", qo.msg.c_str());
        if (isrep[a]) {
          std::vector<std::pair<uint32_t, uint64_t>> spill;
          for (uint64_t off = 0; off < ent; off += mq) {
            const uint64_t len = std::min(mq, ent - off);
            piece_rp[0] = 0;
            piece_rp[1] = len;
            piece_rp[2] = 0;
            if (int r = hc.h2d(D.rp, piece_rp.data(), 16)) return r;
            if (int r = hc.h2d(D.qoff, piece_rp.data() + 2, 8)) return r;
            HIP_TRY(hipStreamSynchronize(s));
            if (int r = hc.h2d(D.col, G.col + ea + off, 4 * len)) return r;
            if (G.wt)
              if (int r = hc.h2d(D.wt, G.wt + ea + off, 4 * len)) return r;
            wl_csr sg{};
            sg.n = len;
            sg.nnz = 0;
            sg.row_ptr64 = D.rp;
            Session S;
            if (int r = open_session(S, &sg, nullptr, W + QL.core, QL.total - QL.core, s))
              return r;
            S.ctx.keys_mat = 1;
            if (int r = S.init_state(0, 1, 0, 1, 1)) return r;
            hipLaunchKernelGGL(k_q_keys, dim3(grid_for(len, kBlock, 8192)), dim3(kBlock), 0, s,
                               S.ctx, D.rp, D.col, G.wt ? D.wt : nullptr, blk_dev, isrep_dev,
                               D.qoff, 1u, (uint32_t)a, blk[a]);
            HIP_LAUNCH_CHECK();
            if (int r = quotient_chunk(S, hc, D, len, 1, blk[a], ea + ent, Q, &spill, hkey, hw,
                                       hdeg))
              return r;
          }
          std::sort(spill.begin(), spill.end());
          for (size_t i = 0; i < spill.size();) {
            size_t k2 = i;
            uint64_t w = 0;
            while (k2 < spill.size() && spill[k2].first == spill[i].first) w += spill[k2++].second;
            if (w > 0xFFFFFFFFull) return fail(WL_EOVERFLOW, "a quotient weight exceeds 2^32 - 1");
            if (Q.m >= std::min(Q.cap, ea + ent))
              return fail(WL_EINVAL, "quotient larger than expected");
            Q.deg[blk[a]] += 1;
            Q.col[Q.m] = spill[i].first;
            Q.wt[Q.m] = (uint32_t)w;
            Q.m++;
            i = k2;
          }
        }
        push_job({j, 0, 0, 0, 0, false});
      } else if (qs[st].run > 0) {
        const QChunkPrep& q = qs[st];
        const uint64_t nrows = c.bnd - a;
        clk::time_point tq = clk::now();
        ++q_chunks;
        HIP_TRY(hipStreamWaitEvent(s, qp.ready[st], 0));
        wl_csr sg{};
        sg.n = q.run;
        sg.nnz = 0;
        sg.row_ptr64 = D.rp;
        Session S;
        if (int r = open_session(S, &sg, nullptr, W + QL.core, QL.total - QL.core, s))
          return r;
        S.ctx.keys_mat = 1;
        if (int r = S.init_state(0, 1, 0, 1, 1)) return r;
        hipLaunchKernelGGL(k_q_keys, dim3(grid_for(ent, kBlock, 8192)),
                           dim3(kBlock), 0, s, S.ctx, D.rp, D.col,
                           G.wt ? D.wt : nullptr, blk_dev, isrep_dev, D.qoff,
                           (uint32_t)nrows, (uint32_t)a, q.bfirst);
        HIP_LAUNCH_CHECK();
        uint64_t nd = 0;
        if (int r = quotient_chunk(S, hc, D, q.run, q.nreps, q.bfirst, ea + ent, Q, nullptr,
                                   hkey, hw, hdeg, &q.qseg, trace ? q_tm : nullptr, &nd))
          return r;
        if (trace) q_dev_ms += ms_since(tq);
        push_job({j, nd, q.nreps, ea + ent, q.bfirst, true});
      } else {
        push_job({j, 0, 0, 0, 0, false});
      }
      // the device must not start chunk j+1 before the copies out of chunk
      // j-1 (its input set) are done: the prefetcher waits for that; a
      // failed copy ends the loop here
      {
        std::lock_guard<std::mutex> g(qo.m);
        if (qo.err != WL_OK) return fail(qo.err, "%s", qo.msg.c_str());
      }
    }
    if (wait_out(qch.size())) return fail(qo.err, "%s", qo.msg.c_str());
    qp.th.join();
    if (qp.err != WL_OK) return fail(qp.err, "%s", qp.msg.c_str());
    if (trace) {
      fprintf(stderr, "[wl batched] t=%llu quotient: %llu chunks, waiting for copies in, device "
              "and copies out %.1f ms (device %.1f, out %.1f), %.1f ms since the last line\n",
              (unsigned long long)t, (unsigned long long)q_chunks, q_dev_ms, q_tm[0], q_tm[1],
              ms_since(t_phase));
      t_phase = clk::now();
    }
    // new row pointers and labels
    if (int r = nrp_buf.alloc(8 * (nq + 1))) return r;
    uint64_t* qrp = nrp_buf.as<uint64_t>();
    qrp[0] = 0;
    for (uint64_t q = 0; q < nq; ++q) qrp[q + 1] = qrp[q] + Q.deg[q];
    if (!labels.empty()) {
      std::vector<uint32_t> nl(nq);
      for (uint64_t i = 0; i < n; ++i)
        if (isrep[i]) nl[blk[i]] = labels[i];
      labels.swap(nl);
    }
    std::swap(qrp_buf.p, nrp_buf.p);
    nrp_buf.p.reset();
    if (!in_place) {
      std::swap(qcol_buf.p, ncol_buf.p);
      std::swap(qwt_buf.p, nwt_buf.p);
    }
    G.n = nq;
    G.m = Q.m;
    G.rp32 = nullptr;
    G.rp64 = qrp_buf.as<const uint64_t>();
    G.col = qcol_buf.as<const uint32_t>();
    G.wt = qwt_buf.as<const uint32_t>();
    if (int r = plan_batches(G, &mb, &starts)) return r;
    // Section 5.4's termination: stop when the next iteration would not
    // have fewer batches
    if (early && starts.size() - 1 >= nb) {
      if (exact) return finish_exact(G);
      *coarsest_out = 0;
      break;
    }
  }
  // final colours: first occurrence over the original nodes
  canonical_colours(map0, nullptr, G.n, color_out, k_out);
  *rounds_out = (uint32_t)std::min<uint64_t>(rounds, 0xFFFFFFFFull);
  *outer_out = outer;
  return WL_OK;
}

