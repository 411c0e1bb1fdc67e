// Host driver and C ABI (include/wl.h) of the gfx950 path.
//
// Algorithm 1 (Section 4.1): each round is
//   x_i = W(seed, r, c_i)  ->  z = A x (mod p)  ->  relabel by (c_i, z_i)
// and rounds repeat until the colour count is unchanged.  The library keeps
// the nodes grouped by colour between rounds, skips singleton classes, and
// never allocates: every buffer is carved from the caller's workspace.
#include <hip/hip_runtime.h>

#include <sched.h>

#include <algorithm>
#include <chrono>
#include <condition_variable>
#include <deque>
#include <functional>
#include <mutex>
#include <string>
#include <memory>
#include <new>
#include <thread>
#include <type_traits>
#include <utility>
#include <vector>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../include/wl.h"
#include "wl_host.h"
#include "wl_ctx.h"
#include "wl_relabel.h"
#include "wl_live.h"
#include "wl_degree.h"
#include "wl_stream.h"
#include "wl_spmv.h"
#include "wl_push.h"
#include "wl_quotient.h"
#include "wl_verify.h"

using namespace wl;

namespace {

thread_local char g_err[512] = "";
thread_local int g_stats_flags = 0;
thread_local wl_stats g_stats{};
// Arithmetic of the image step on this thread (wl_set_precision): 0 = F_p,
// 1 = Z/2^64.
thread_local uint32_t g_ring = 0;

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

#define HIP_TRY(expr)                                                      \
  do {                                                                     \
    hipError_t e_ = (expr);                                                \
    if (e_ != hipSuccess)                                                  \
      return fail(WL_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define HIP_LAUNCH_CHECK()                                                    \
  do {                                                                        \
    hipError_t e_ = hipGetLastError();                                        \
    if (e_ != hipSuccess)                                                     \
      return fail(WL_EHIP, "kernel launch failed: %s", hipGetErrorString(e_)); \
  } while (0)

constexpr uint64_t kAlign = 256;
// Largest input of wl_stable_coloring_batched with WL_BATCHED_EXACT.
constexpr uint64_t kExactFinishMaxEntries = 1ull << 31;
uint64_t align_up(uint64_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Sizes of every workspace region for a graph with n nodes, nnz entries.
// in_core = false: a session whose image is computed elsewhere (the streamed
// rounds), without the SpMV schedule and the live-class state.
struct Layout {
  uint64_t n, nnz;
  uint32_t max_small, max_big, max_chunks, max_heavy;
  bool in_core;
  uint64_t off_st, off_x, off_z, off_keys, off_keys_tmp, off_perm, off_perm_tmp,
      off_ids, off_cstart, off_flags, off_act, off_small, off_tiny, off_big0, off_big1,
      off_tile, off_bhist, off_bmin, off_bmax, off_bcur, off_scan, off_rows,
      off_binpart, off_chunks, off_hacc, off_hcnt, off_wtab, off_c16, off_qcls2, off_lcls[2],
      off_rs[2], off_rl[2], off_hq, off_bsame, off_nz0f, off_pos, off_desc;
  uint32_t desc_cap;  // chunks of a chained scan (kBlock live classes, or more items)
  uint64_t total;
};

Layout make_layout(uint64_t n, uint64_t nnz, bool in_core = true) {
  Layout L{};
  const uint64_t nc = in_core ? n : 0;
  L.in_core = in_core;
  L.n = n;
  L.nnz = nnz;
  L.max_small = (uint32_t)(n / 2 + 1);
  L.max_big = (uint32_t)(n / (kSmallMax + 1) + 1);
  L.max_heavy = (uint32_t)std::min<uint64_t>(n, nnz / (kHeavyChunk + 1) + 1);
  L.max_chunks = (uint32_t)(nnz / kHeavyChunk + L.max_heavy + 1);
  uint64_t o = 0;
  auto take = [&](uint64_t bytes) {
    uint64_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L.off_st = take(sizeof(DevState));
  L.off_x = take(8 * n);
  L.off_z = take(8 * n);
  L.off_keys = take(8 * n);
  L.off_keys_tmp = take(8 * n);
  L.off_perm = take(4 * n);
  L.off_perm_tmp = take(4 * n);
  L.off_ids = take(4 * (n + 1));
  L.off_cstart = take(4 * (n + 2));
  L.off_flags = take(n + 1);
  L.off_act = take(n + 1);
  L.off_small = take(8ull * (n / (kTinyMax + 1) + 1));
  L.off_tiny = take(8ull * L.max_small);
  L.off_big0 = take(8ull * L.max_big);
  L.off_big1 = take(8ull * L.max_big);
  L.off_tile = take(8ull * (L.max_big + 1));
  L.off_bhist = take(4ull * L.max_big * kRadix);
  L.off_bmin = take(8ull * L.max_big * kRadix);
  L.off_bmax = take(8ull * L.max_big * kRadix);
  L.off_bcur = take(4ull * L.max_big * kRadix);
  L.off_scan = take(8ull * kScanBlocks);
  L.off_rows = take(4 * nc);
  L.off_binpart = take(4ull * kNumBins * kScanBlocks);
  L.off_chunks = take(in_core ? sizeof(HeavyChunk) * (uint64_t)L.max_chunks : 0);
  L.off_hacc = take(in_core ? 16ull * L.max_heavy : 0);
  L.off_hcnt = take(in_core ? 4ull * L.max_heavy : 0);
  L.off_wtab = take(8ull * std::min<uint64_t>(n, kTableMax));
  L.off_c16 = take(2 * n);
  L.off_qcls2 = take(4 * nc);
  // live classes have >= 2 members: at most n / 2 of them, three words each
  L.off_lcls[0] = take(in_core ? 12ull * (n / 2 + 1) : 0);
  L.off_lcls[1] = take(in_core ? 12ull * (n / 2 + 1) : 0);
  L.off_rs[0] = take(8 * nc);
  L.off_rs[1] = take(8 * nc);
  L.off_rl[0] = take(4 * nc);
  L.off_rl[1] = take(4 * nc);
  L.off_hq = take(in_core ? 4ull * L.max_heavy : 0);
  L.off_bsame = take(L.max_big + 1);
  L.off_nz0f = take(in_core ? n + 1 : 0);
  L.off_pos = take(in_core ? 4ull * n : 0);
  L.desc_cap = (uint32_t)(n / kBlock + 2);
  L.off_desc = take(in_core ? 16ull * L.desc_cap : 0);
  L.total = o;
  return L;
}

// Workspace of the propagation-blocking image (symmetric unweighted graphs
// with fewer than 2^32 entries), placed after the in-core layout.  Offsets
// are relative to its start.
struct PbLayout {
  bool ok = false;
  uint32_t levels = 0, shift1 = 0, nb1 = 0, nfine = 0, fbits = 0;
  uint64_t ntiles1 = 0;
  uint64_t cnt = 0, bstart1 = 0, bstartf = 0, rec1 = 0, rec2 = 0, tile_row = 0,
           tile2_off = 0, cur1 = 0, cur2 = 0, slice_off = 0, mslice_off = 0, mlist = 0,
           part = 0;
  uint64_t total = 0;
};

PbLayout make_pb_layout(uint64_t n, uint64_t nnz) {
  PbLayout P{};
  if (n == 0 || nnz == 0 || nnz >= (1ull << 32) || n >= (1ull << 32) - (1ull << 16)) return P;
  const uint64_t nf = (n + kPbFineRows - 1) >> kPbFineShift;
  P.nfine = (uint32_t)nf;
  if (nf <= kPbMaxBins) {
    P.levels = 1;
    P.shift1 = kPbFineShift;
  } else {
    uint32_t fb = 0;
    while (((nf + (1ull << fb) - 1) >> fb) > kPbMaxBins) ++fb;
    if ((1u << fb) > kPbMaxFine) return P;  // pass 2 splits a coarse bin at most this far
    P.levels = 2;
    P.fbits = fb;
    P.shift1 = kPbFineShift + fb;
  }
  P.nb1 = (uint32_t)((n + (1ull << P.shift1) - 1) >> P.shift1);
  P.ntiles1 = (nnz + kPbTile - 1) / kPbTile;
  // slices of the bins cut into several: each holds more than kPbSlice
  // records, so together fewer than 2 * nnz / kPbSlice
  const uint64_t mslots = 2 * ((nnz + kPbSlice - 1) / kPbSlice) + 1;
  uint64_t o = 0;
  auto take = [&](uint64_t bytes) {
    uint64_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  P.cnt = take(sizeof(PbCounts));
  P.bstart1 = take(8ull * (P.nb1 + 1));
  P.bstartf = take(8 * (nf + 1));
  P.rec1 = take(P.levels == 2 ? 4 * nnz : 0);
  P.rec2 = take(4 * nnz);
  P.tile_row = take(4 * P.ntiles1);
  P.tile2_off = take(4ull * (P.nb1 + 1));
  P.cur1 = take(8ull * P.nb1);
  P.cur2 = take(8 * nf);
  P.slice_off = take(4 * (nf + 1));
  P.mslice_off = take(4 * (nf + 1));
  P.mlist = take(4 * nf);
  P.part = take(8ull * kPbFineRows * mslots);
  P.total = o;
  P.ok = true;
  return P;
}

// The Ctx of a live round whose current lists are the other buffer set: the
// '2' arrays become current and the current ones receive the next round's
// lists (so no copy is needed between rounds).  lperm is the sort's payload,
// so perm and perm_tmp swap with it; the per-round wave queue lives in the
// buffer that is not current.
Ctx swapped_live(const Ctx& c) {
  Ctx x = c;
  std::swap(x.perm, x.perm_tmp);
  std::swap(x.lperm, x.lperm2);
  std::swap(x.qcls, x.qcls2);
  x.midq = x.qcls2;
  std::swap(x.lcold, x.lcold2);
  std::swap(x.loff, x.loff2);
  std::swap(x.llen, x.llen2);
  std::swap(x.rs, x.rs2);
  std::swap(x.rl, x.rl2);
  return x;
}

bool wants_pb(const wl_csr* g) {
  return (g->flags & WL_CSR_SYMMETRIC) && g->weight == nullptr;
}

Ctx make_ctx(const Layout& L, const wl_csr* g, uint8_t* ws, uint32_t* colors) {
  Ctx c{};
  c.ring = g_ring;
  c.n = (uint32_t)L.n;
  c.nnz = L.nnz;
  c.rp32 = g->row_ptr32;
  c.rp64 = g->row_ptr64;
  c.col = g->col_idx;
  c.wgt = g->weight;
  c.st = (DevState*)(ws + L.off_st);
  c.c = colors;
  c.x = (uint64_t*)(ws + L.off_x);
  c.z = (uint64_t*)(ws + L.off_z);
  c.keys = (uint64_t*)(ws + L.off_keys);
  c.keys_tmp = (uint64_t*)(ws + L.off_keys_tmp);
  c.perm = (uint32_t*)(ws + L.off_perm);
  c.perm_tmp = (uint32_t*)(ws + L.off_perm_tmp);
  c.ids = (uint32_t*)(ws + L.off_ids);
  c.cstart = (uint32_t*)(ws + L.off_cstart);
  c.flags = ws + L.off_flags;
  c.act = ws + L.off_act;
  c.small_list = (uint2*)(ws + L.off_small);
  c.tiny_list = (uint2*)(ws + L.off_tiny);
  c.big_list0 = (uint2*)(ws + L.off_big0);
  c.big_list1 = (uint2*)(ws + L.off_big1);
  c.tile_off0 = (uint32_t*)(ws + L.off_tile);
  c.tile_off1 = c.tile_off0 + L.max_big + 1;
  c.bhist = (uint32_t*)(ws + L.off_bhist);
  c.bmin = (unsigned long long*)(ws + L.off_bmin);
  c.bmax = (unsigned long long*)(ws + L.off_bmax);
  c.bcur = (uint32_t*)(ws + L.off_bcur);
  c.scan_part = (uint32_t*)(ws + L.off_scan);
  c.rows = (uint32_t*)(ws + L.off_rows);
  c.bin_part = (uint32_t*)(ws + L.off_binpart);
  c.chunks = (HeavyChunk*)(ws + L.off_chunks);
  c.hacc = (unsigned long long*)(ws + L.off_hacc);
  c.hcnt = (uint32_t*)(ws + L.off_hcnt);
  c.wtab = (uint64_t*)(ws + L.off_wtab);
  c.c16 = (uint16_t*)(ws + L.off_c16);
  c.c8 = ws + L.off_c16;
  // Live-class state.  The incremental rounds do not use the full relabel's
  // grouping (perm, cstart), its flags, x, or keys_tmp/tiny_list outside the
  // sort, so those regions are shared:
  //   lperm = perm (the sort's payload), lperm2 = perm_tmp (the sort's
  //   scratch, written after it), qcls = cstart, gnz = flags, gl/go = x,
  //   gstart/gend = keys_tmp, split = tiny_list, shift = keys (written after
  //   the last read of keys).
  c.lperm = c.perm;
  c.lperm2 = c.perm_tmp;
  c.qcls = c.cstart;
  c.qcls2 = (uint32_t*)(ws + L.off_qcls2);
  {
    const uint64_t m = L.n / 2 + 1;
    uint32_t* a = (uint32_t*)(ws + L.off_lcls[0]);
    uint32_t* b = (uint32_t*)(ws + L.off_lcls[1]);
    c.lcold = a;
    c.loff = a + m;
    c.llen = a + 2 * m;
    c.lcold2 = b;
    c.loff2 = b + m;
    c.llen2 = b + 2 * m;
  }
  c.gnz = c.flags;
  c.gl = (uint32_t*)c.x;
  c.go = (uint32_t*)c.x + L.n;
  c.gstart = (uint32_t*)c.keys_tmp;
  c.gend = (uint32_t*)c.keys_tmp + L.n;
  c.split = c.tiny_list;
  c.shift = (uint32_t*)c.keys;
  c.rs = (uint64_t*)(ws + L.off_rs[0]);
  c.rs2 = (uint64_t*)(ws + L.off_rs[1]);
  c.rl = (uint32_t*)(ws + L.off_rl[0]);
  c.rl2 = (uint32_t*)(ws + L.off_rl[1]);
  c.midq = c.qcls2;  // consumed by the SpMV before k_live_emit writes qcls2
  c.hq = (uint32_t*)(ws + L.off_hq);
  c.bsame = ws + L.off_bsame;
  c.nz0f = L.in_core ? ws + L.off_nz0f : nullptr;
  c.pos = L.in_core ? (uint32_t*)(ws + L.off_pos) : nullptr;
  c.pos_deg = c.pos;
  c.desc = L.in_core ? (unsigned long long*)(ws + L.off_desc) : nullptr;
  c.desc_cap = L.desc_cap;
  c.lsplit = c.c8;    // the live rounds do not use the compact colours
  c.weighted = g->weight != nullptr;
  {
    const char* nt = getenv("WL_NT_STREAM");
    c.nt_stream = nt && nt[0] == '1';
  }
  {
    // WL_SORT_FIX=0 sends every small segment with a mixed bucket to the
    // sorting network (the tests use it to run that path)
    const char* f = getenv("WL_SORT_FIX");
    const long v = f ? strtol(f, nullptr, 10) : (long)kCsFix;
    c.cs_fix = (uint32_t)std::min<long>(std::max<long>(v, 0), (long)kSmallMax);
  }
  {
    // WL_CHAIN_SPINS=n bounds the wait of a chained scan for an earlier chunk
    // (the tests make it tiny to run the give-up path: the call then fails
    // with WL_EHIP, or completes when no wait was needed)
    const char* f = getenv("WL_CHAIN_SPINS");
    const long v = f ? strtol(f, nullptr, 10) : (long)kChainSpins;
    c.chain_spins = (uint32_t)std::min<long>(std::max<long>(v, 0), (long)kChainSpins);
  }
  c.max_small = L.max_small;
  c.max_sm = (uint32_t)(L.n / (kTinyMax + 1) + 1);
  c.max_big = L.max_big;
  c.max_chunks = L.max_chunks;
  c.max_heavy = L.max_heavy;
  return c;
}

uint32_t grid_for(uint64_t work, uint32_t per_block = kBlock,
                  uint32_t cap = 8192) {
  uint64_t b = (work + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (uint32_t)b;
}

uint32_t scan_blocks(uint64_t n) {
  uint64_t b = (n + 4 * kBlock - 1) / (4 * kBlock);
  return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(b, kScanBlocks));
}

int check_graph(const wl_csr* g) {
  if (!g) return fail(WL_EINVAL, "graph is NULL");
  if (g->n >= (1ull << 32))
    return fail(WL_EOVERFLOW, "n = %llu does not fit 32-bit node ids",
                (unsigned long long)g->n);
  if ((g->row_ptr32 == nullptr) == (g->row_ptr64 == nullptr))
    return fail(WL_EINVAL, "exactly one of row_ptr32/row_ptr64 must be set");
  if (g->row_ptr32 && g->nnz >= (1ull << 32))
    return fail(WL_EINVAL, "nnz >= 2^32 needs row_ptr64");
  if (g->nnz > 0 && g->col_idx == nullptr)
    return fail(WL_EINVAL, "col_idx is NULL");
  return WL_OK;
}

// Reads row_ptr[n] from the device and compares it with nnz.
int check_nnz_device(const wl_csr* g, hipStream_t s) {
  uint64_t last = 0;
  if (g->row_ptr32) {
    uint32_t v = 0;
    HIP_TRY(hipMemcpyAsync(&v, g->row_ptr32 + g->n, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    last = v;
  } else {
    HIP_TRY(hipMemcpyAsync(&last, g->row_ptr64 + g->n, 8, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
  }
  if (last != g->nnz)
    return fail(WL_EINVAL, "row_ptr[n] = %llu but nnz = %llu",
                (unsigned long long)last, (unsigned long long)g->nnz);
  return WL_OK;
}

// ---------------------------------------------------------------------------
// Device-side validation (WL_VALIDATE=1) and small set-up kernels.
// ---------------------------------------------------------------------------

template <typename RP>
__global__ void __launch_bounds__(kBlock) k_validate(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  for (uint64_t i = blockIdx.x * (uint64_t)kBlock + threadIdx.x; i < ctx.n;
       i += (uint64_t)gridDim.x * kBlock)
    if (rp[i + 1] < rp[i]) atomicOr(&ctx.st->err, 1u);
  for (uint64_t e = blockIdx.x * (uint64_t)kBlock + threadIdx.x; e < ctx.nnz;
       e += (uint64_t)gridDim.x * kBlock)
    if (ctx.col[e] >= ctx.n) atomicOr(&ctx.st->err, 2u);
}

// Symmetry of a graph flagged WL_CSR_SYMMETRIC (validation only): the sums
// over all entries of a 64-bit hash of (row, column) and of (column, row)
// agree exactly when the two multisets of entries are equal, up to a hash
// collision.
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_validate_sym(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  unsigned long long f = 0, b = 0;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n; i += gridDim.x * kBlock)
    for (uint64_t e = rp[i]; e < rp[i + 1]; ++e) {
      const uint64_t j = ctx.col[e];
      const uint64_t w = ctx.wgt ? ctx.wgt[e] : 1u;
      f += mix64(mix64(((uint64_t)i << 32) | j) + w);
      b += mix64(mix64((j << 32) | i) + w);
    }
  atomicAdd(&ctx.st->sym_hash[0], f);
  atomicAdd(&ctx.st->sym_hash[1], b);
}

constexpr uint32_t kErrRowSum = 32u;  // DevState::err bit: a row sum above 2^32 (ring)

// Theorem 1's precondition for Z/2^64: every row sum of A at most 2^32.  One
// thread per row (its length, or the sum of at most 64 weights); the rows
// with more weights are summed by all 64 lanes of the wave, one after the
// other.  Sets kErrRowSum on a row above the bound.
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_ring_rows(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t lane = lane_id();
  const uint64_t lim = 1ull << 32;
  // 'base' is the same for all lanes of a wave, so every lane runs every
  // iteration (the shuffles below need the whole wave)
  for (uint64_t base = blockIdx.x * (uint64_t)kBlock + threadIdx.x - lane; base < ctx.n;
       base += (uint64_t)gridDim.x * kBlock) {
    const uint64_t i = base + lane;
    uint64_t beg = 0, end = 0;
    if (i < ctx.n) {
      beg = rp[i];
      end = rp[i + 1];
    }
    bool over = false, wide = false;
    if (!ctx.wgt) {
      over = end - beg > lim;
    } else if (end - beg <= (uint64_t)kWave) {
      uint64_t sum = 0;
      for (uint64_t e = beg; e < end; ++e) sum += ctx.wgt[e];
      over = sum > lim;
    } else {
      wide = true;
    }
    for (uint64_t m = __ballot(wide); m; m &= m - 1) {
      const int l = __builtin_ctzll(m);
      const uint64_t b = read_lane64(beg, l), e = read_lane64(end, l);
      uint64_t sum = 0;
      for (uint64_t x = b + lane; x < e; x += kWave) sum += ctx.wgt[x];
      for (int off = kWave / 2; off > 0; off >>= 1) sum += __shfl_xor(sum, off, kWave);
      if (sum > lim) over = true;
    }
    if (over) atomicOr(&ctx.st->err, kErrRowSum);
  }
}

__global__ void __launch_bounds__(kBlock) k_check_colors(Ctx ctx,
                                                         const uint32_t* col,
                                                         uint32_t k) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock)
    if (col[i] >= k) atomicOr(&ctx.st->err, 4u);
}

__global__ void __launch_bounds__(kBlock) k_iota_zero(Ctx ctx) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock) {
    ctx.perm[i] = i;
    ctx.ids[i] = 0;
    ctx.c[i] = 0;
    ctx.act[i] = ctx.n >= 2 ? 1 : 0;
    if (ctx.nz0f) ctx.nz0f[i] = 0;
  }
  // chained-scan descriptors: nothing left from an earlier call may read as
  // ready (their epochs restart with the rounds)
  if (ctx.desc)
    for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < 2 * ctx.desc_cap;
         i += gridDim.x * kBlock)
      ctx.desc[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctx.cstart[0] = 0;
    ctx.cstart[1] = ctx.n;
  }
}

__global__ void __launch_bounds__(kBlock) k_labels_to_z(Ctx ctx,
                                                        const uint32_t* lab) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock)
    ctx.z[i] = lab[i];
}

// Counting sort of the nodes by colour (colours < k): cstart, perm, act.
__global__ void __launch_bounds__(kBlock) k_count_colors(Ctx ctx, uint32_t k) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i <= k;
       i += gridDim.x * kBlock)
    ctx.ids[i] = 0;
}
// Class sizes of a given colouring.  The lanes of a wave that share a colour
// add their count with one atomic (a colouring with few classes would
// otherwise put most atomics of the device on one address).
__global__ void __launch_bounds__(kBlock) k_hist_colors(Ctx ctx) {
  const uint32_t lane = lane_id();
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock) {
    const uint32_t c = ctx.c[i];
    const unsigned long long peers = wave_peers(c, true);
    if ((int)lane == __ffsll((long long)peers) - 1)
      atomicAdd(&ctx.ids[c], (uint32_t)__popcll(peers));
  }
}
// One block: cstart = exclusive scan of ids[0..k]; ids becomes the cursor.
__global__ void __launch_bounds__(kBlock) k_scan_colors(Ctx ctx, uint32_t k) {
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t carry = 0;
  for (uint32_t base = 0; base <= k; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i <= k ? ctx.ids[i] : 0;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(v, sh, &tot);
    if (i <= k) {
      ctx.cstart[i] = carry + ex;
      ctx.ids[i] = carry + ex;
    }
    carry += tot;
  }
}
// Nodes grouped by colour: one cursor reservation per colour present in a
// wave, the lanes' slots by their position among its peers.
__global__ void __launch_bounds__(kBlock) k_place_colors(Ctx ctx) {
  const uint32_t lane = lane_id();
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock) {
    const uint32_t c = ctx.c[i];
    const unsigned long long peers = wave_peers(c, true);
    const int ldr = __ffsll((long long)peers) - 1;
    uint32_t at = 0;
    if ((int)lane == ldr) at = atomicAdd(&ctx.ids[c], (uint32_t)__popcll(peers));
    at = __shfl(at, ldr, kWave) + (uint32_t)__popcll(peers & ((1ull << lane) - 1));
    ctx.perm[at] = i;
    ctx.act[i] = (ctx.cstart[c + 1] - ctx.cstart[c]) >= 2 ? 1 : 0;
  }
}

// ---------------------------------------------------------------------------
// One call's device session.
// ---------------------------------------------------------------------------

constexpr uint32_t kHostRounds = 8;
constexpr int kAsyncPassesDefault = 2;

int env_int(const char* name, int lo, int hi, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  const int x = atoi(v);
  return x < lo ? lo : (x > hi ? hi : x);
}

struct Session {
  Layout L;
  Ctx ctx;
  // Rounds driven from the host before device-driven groups start, and radix
  // passes a device-driven round runs before it halts for the host.  Both
  // can be set for testing (WL_HOST_ROUNDS, WL_ASYNC_PASSES).
  uint32_t host_rounds_first = kHostRounds;
  int async_passes = kAsyncPassesDefault;
  int passes_seen = 0;      // most radix passes a host-driven sort needed
  // Live rounds alternate between two buffer sets: round r reads the set
  // (r - live_r0) & 1 and writes the other; ctx0 has set 0 current.
  Ctx ctx0{};
  uint32_t live_r0 = 0;
  bool hist_clean = false;  // radix histograms cleared (first pass of the call)
  hipStream_t s;
  bool rp64;
  bool weighted;
  // Propagation blocking (symmetric graphs): available when the workspace
  // holds its layout; planned at its first use; stopped for the rest of the
  // call once fewer than half of the entries feed rows whose image is needed
  // (that fraction never grows).  WL_PB=0 turns it off, WL_PB=force uses it
  // in every round it can serve (for testing).
  PbLayout P;
  PbCtx pb{};
  uint32_t live_heavy = 0, live_mid = 0;  // blocks of k_spmv_mid
  bool live_mode = false;                  // incremental rounds (run_rsc)
  bool live_built = false;                 // live classes set up
  // The one-colour round by degree histogram (WL_DEGREE_ROUND=0 turns it off,
  // for testing the general path).
  bool deg_mode = true;
  PbCounts pbc{};
  bool pb_avail = false, pb_planned = false, pb_stop = false;
  // pos_deg holds the member-list positions of the coming round's live
  // classes (set by the one-colour round, cleared by the next image)
  bool deg_pos_fresh = false;
  bool sym_flag = false;
  int pb_mode = 1;
  DevState host;      // last copy of the device state
  DevState init_src;  // source of the initial state copy
  uint32_t nscan;
  // diagnostics: SpMV launches bracketed by events, folded in at the next
  // read-back (a launch queued for a round that never ran is dropped)
  struct TimedSpmv {
    hipEvent_t a, b;
    uint32_t round;  // the round it belongs to
    bool always;     // launched by a host-driven round: it ran
    int kind;        // kImgGather, kImgPb, kImgUniform
  };
  int sflags = 0;
  hipEvent_t call_ev[2] = {nullptr, nullptr};
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<TimedSpmv> timed;
  wl_stats stats{};

  // WL_GRAPH=1: device-driven rounds replayed from a HIP graph of two rounds
  // (one per buffer-set parity of its first round), captured on a stream of
  // the session's own.  Off by default: on the 1024 x 1024 grid (512 rounds)
  // replay took 277 ms against 132 ms for the same kernels launched on the
  // stream.
  bool use_graph = false;
  bool capturing = false;
  hipStream_t cap_stream = nullptr;
  hipGraphExec_t gexec[2] = {nullptr, nullptr};
  int gexec_ap[2] = {-1, -1};  // radix passes per round when captured

  ~Session() {
    for (hipEvent_t& e : call_ev)
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t& e : ev_pool) (void)hipEventDestroy(e);
    for (hipGraphExec_t& g : gexec)
      if (g) (void)hipGraphExecDestroy(g);
    if (cap_stream) (void)hipStreamDestroy(cap_stream);
  }

  int stats_begin() {
    sflags = g_stats_flags;
    stats = wl_stats{};
    if (sflags & WL_STATS_TIME) {
      for (hipEvent_t& e : call_ev) HIP_TRY(hipEventCreate(&e));
      HIP_TRY(hipEventRecord(call_ev[0], s));
    }
    return WL_OK;
  }

  // Timing-only events: read after a synchronising read-back, so they take
  // no system-scope fence (whose cache write-back and invalidation would
  // slow the launches that follow each record).
  hipEvent_t next_event() {
    if (ev_used == ev_pool.size()) {
      hipEvent_t e = nullptr;
      if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
      ev_pool.push_back(e);
    }
    return ev_pool[ev_used++];
  }

  // Brackets the launches issued by 'launch' with events when timing is on;
  // launches are counted when the round is known to have run.
  template <typename F>
  void timed_spmv(uint32_t round, bool always, int kind, F&& launch) {
    if (capturing) {  // replayed launches are not timed
      launch();
      return;
    }
    TimedSpmv t{nullptr, nullptr, round, always, kind};
    if (sflags & WL_STATS_TIME) {
      t.a = next_event();
      t.b = next_event();
    }
    if (t.a && t.b) (void)hipEventRecord(t.a, s);
    launch();
    if (t.a && t.b) (void)hipEventRecord(t.b, s);
    timed.push_back(t);
  }

  // after a synchronising pull
  int stats_collect() {
    const uint32_t ran =
        host.round + (host.done == kHalted || host.done == kHaltedShift ? 1u : 0u);
    for (const TimedSpmv& t : timed) {
      if (!t.always && t.round >= ran) continue;
      float ms = 0;
      if (t.a && t.b) HIP_TRY(hipEventElapsedTime(&ms, t.a, t.b));
      wl_stats_kind& sk = t.kind == kImgPb ? stats.pb
                          : (t.kind == kImgUniform ? stats.uniform : stats.gather);
      sk.ms += ms;
      sk.launches++;
    }
    timed.clear();
    ev_used = 0;
    return WL_OK;
  }

  int stats_end() {
    if (sflags & WL_STATS_TIME) {
      HIP_TRY(hipEventRecord(call_ev[1], s));
      HIP_TRY(hipEventSynchronize(call_ev[1]));
      float ms = 0;
      HIP_TRY(hipEventElapsedTime(&ms, call_ev[0], call_ev[1]));
      stats.call_ms = ms;
    }
    if (int r = pull()) return r;
    stats.rounds = host.round;
    stats.gather.rows = host.work[kImgGather][0];
    stats.gather.entries = host.work[kImgGather][1];
    stats.pb.rows = host.work[kImgPb][0];
    stats.pb.entries = host.work[kImgPb][1];
    stats.uniform.rows = host.work[kImgUniform][0];
    stats.uniform.entries = host.work[kImgUniform][1];
    g_stats = stats;
    return WL_OK;
  }

  int pull() {
    HIP_TRY(hipMemcpyAsync(&host, ctx.st, sizeof(DevState), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return stats_collect();
  }

  // The source of the copy is a member that outlives it, and the copy is
  // synchronised: an asynchronous copy from pageable host memory may read
  // the source after this function returns.
  int init_state(uint64_t seed, uint32_t k, uint32_t round, uint32_t max_rounds,
                 uint32_t dense) {
    DevState h{};
    h.k = k;
    h.dense = dense;
    h.round = round;
    h.max_rounds = max_rounds;
    h.seed = seed;
    host = h;
    init_src = h;
    HIP_TRY(hipMemcpyAsync(ctx.st, &init_src, sizeof(DevState), hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));
    return WL_OK;
  }

  int validate_device() {
    const char* v = getenv("WL_VALIDATE");
    if (!v || v[0] != '1') return WL_OK;
    uint32_t g = grid_for(std::max<uint64_t>(L.n, L.nnz));
    if (rp64)
      hipLaunchKernelGGL(k_validate<uint64_t>, dim3(g), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_validate<uint32_t>, dim3(g), dim3(kBlock), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    if (host.err & 1u) return fail(WL_EINVAL, "row_ptr is not non-decreasing");
    if (host.err & 2u) return fail(WL_EINVAL, "a column index is >= n");
    if (sym_flag) {
      if (rp64)
        hipLaunchKernelGGL(k_validate_sym<uint64_t>, dim3(grid_for(L.n)), dim3(kBlock), 0, s, ctx);
      else
        hipLaunchKernelGGL(k_validate_sym<uint32_t>, dim3(grid_for(L.n)), dim3(kBlock), 0, s, ctx);
      HIP_LAUNCH_CHECK();
      if (int r = pull()) return r;
      if (host.sym_hash[0] != host.sym_hash[1])
        return fail(WL_EINVAL, "the graph is flagged symmetric but is not");
    }
    return WL_OK;
  }

  // In Z/2^64, Theorem 1's bound on the row sums (n < 2^32 holds already).
  int check_ring() {
    if (!ctx.ring) return WL_OK;
    const uint32_t g = grid_for(L.n, kBlock, 4096);
    if (rp64)
      hipLaunchKernelGGL(k_ring_rows<uint64_t>, dim3(g), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_ring_rows<uint32_t>, dim3(g), dim3(kBlock), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    if (host.err & kErrRowSum)
      return fail(WL_EOVERFLOW, "a row sum exceeds 2^32, the bound of arithmetic mod 2^64");
    return WL_OK;
  }

  // The sorting networks (one launch: gt workgroups for the tiny segments,
  // gp for the pico ones, gs for the small ones), with the tie-aware key
  // order in Z/2^64.
  // gs: workgroups of the mid and small sorts (mid segments one per wave)
  void sorts(uint32_t gt, uint32_t gp, uint32_t gs, int check_passes) {
    const uint32_t g = gt + gp + gs;
    if (g == 0) return;
    if (ctx.ring)
      hipLaunchKernelGGL(k_sorts<true>, dim3(g), dim3(kBlock), 0, s, ctx, check_passes, gt, gp);
    else
      hipLaunchKernelGGL(k_sorts<false>, dim3(g), dim3(kBlock), 0, s, ctx, check_passes, gt, gp);
  }

  // SpMV schedule (row bins and heavy chunks); once per call.
  int build_schedule(bool heavy_only = false) {
    const uint32_t nb = scan_blocks(L.n);
    if (rp64)
      hipLaunchKernelGGL(k_bins_count<uint64_t>, dim3(nb), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_bins_count<uint32_t>, dim3(nb), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_bins_scan, dim3(1), dim3(kBlock), 0, s, ctx, nb);
    if (rp64) {
      if (heavy_only)
        hipLaunchKernelGGL((k_bins_fill<uint64_t, true>), dim3(nb), dim3(kBlock), 0, s, ctx);
      else
        hipLaunchKernelGGL((k_bins_fill<uint64_t, false>), dim3(nb), dim3(kBlock), 0, s, ctx);
    } else {
      if (heavy_only)
        hipLaunchKernelGGL((k_bins_fill<uint32_t, true>), dim3(nb), dim3(kBlock), 0, s, ctx);
      else
        hipLaunchKernelGGL((k_bins_fill<uint32_t, false>), dim3(nb), dim3(kBlock), 0, s, ctx);
    }
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    const uint32_t nh = host.bin_cnt[3];
    const uint32_t hb = std::max<uint32_t>(1, std::min<uint32_t>(kScanBlocks, (nh + 255) / 256));
    if (rp64)
      hipLaunchKernelGGL(k_heavy_count<uint64_t>, dim3(hb), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_heavy_count<uint32_t>, dim3(hb), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_heavy_scan, dim3(1), dim3(kBlock), 0, s, ctx, hb);
    if (rp64)
      hipLaunchKernelGGL(k_heavy_fill<uint64_t>, dim3(hb), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_heavy_fill<uint32_t>, dim3(hb), dim3(kBlock), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    return pull();
  }

  template <typename RP, bool W, int M>
  void spmv_launch(const SpmvGrid& g) {
    hipLaunchKernelGGL((k_spmv<RP, W, M>), dim3(g.b0), dim3(kBlock), 0, s, ctx, g);
  }

  // Plan of the propagation-blocking image (once per call).
  template <typename RP>
  int pb_plan() {
    hipLaunchKernelGGL(k_pb_bin_starts<RP>, dim3(grid_for(P.nfine + 1)), dim3(kBlock), 0, s,
                       ctx, pb);
    hipLaunchKernelGGL(k_pb_tile_rows<RP>, dim3(grid_for(L.n, kBlock, 8192)), dim3(kBlock), 0, s,
                       ctx, pb);
    hipLaunchKernelGGL(k_pb_lists<RP>, dim3(1), dim3(kPbThreads), 0, s, ctx, pb);
    HIP_LAUNCH_CHECK();
    HIP_TRY(hipMemcpyAsync(&pbc, pb.cnt, sizeof(PbCounts), hipMemcpyDeviceToHost, s));
    if (int r = pull()) return r;
    pb_planned = true;
    return WL_OK;
  }

  // Whether this round's image goes through propagation blocking: the colour
  // must fit next to the destination in a 32-bit record, and (unless forced)
  // the graph must be large and at least half of its entries must feed rows
  // whose image is needed.
  template <typename RP>
  int pb_wanted(bool* use) {
    *use = false;
    if (!pb_avail || pb_stop || host.k < 2) return WL_OK;
    const uint32_t cbits = 32 - (uint32_t)__builtin_clz(host.k - 1);
    if (P.shift1 + cbits > 32) return WL_OK;
    if (pb_mode == 1) {
      if (L.nnz < kPbMinEntries) {
        pb_stop = true;
        return WL_OK;
      }
      if (live_mode)
        hipLaunchKernelGGL(k_live_count, dim3(grid_for(L.n, kBlock, 4096)), dim3(kBlock), 0, s,
                           ctx, 0);
      else
        hipLaunchKernelGGL(k_count_active<RP>, dim3(grid_for(L.n, kBlock, 4096)), dim3(kBlock),
                           0, s, ctx);
      HIP_LAUNCH_CHECK();
      if (int r = pull()) return r;
      if (host.act_entries * 2 < L.nnz) {
        pb_stop = true;
        return WL_OK;
      }
    }
    pb.cbits = cbits;
    *use = true;
    return WL_OK;
  }

  template <typename RP>
  int pb_round() {
    if (!pb_planned)
      if (int r = pb_plan<RP>()) return r;
    if (sflags & WL_STATS_WORK)
      hipLaunchKernelGGL(k_count_work<RP>, dim3(grid_for(L.n, kBlock, 4096)), dim3(kBlock), 0, s,
                         ctx, kImgPb, 1);
    hipLaunchKernelGGL(k_pb_cursors, dim3(grid_for(P.nfine)), dim3(kBlock), 0, s, ctx, pb);
    timed_spmv(host.round, true, kImgPb, [&] {
      hipLaunchKernelGGL(k_pb_scatter1<RP>, dim3((uint32_t)std::min<uint64_t>(P.ntiles1, 2048)),
                         dim3(kPb1Threads), 0, s, ctx, pb);
      if (P.levels == 2) {
        hipLaunchKernelGGL(k_pb_scatter2, dim3(std::max<uint32_t>(1, pbc.maxtiles2 * P.nb1)),
                           dim3(kPbThreads), 0, s, ctx, pb);
      }
      const dim3 ga(std::max<uint32_t>(1, std::min<uint32_t>(pbc.nslices, 2048)));
      if (host.k <= kPbTableMax)
        hipLaunchKernelGGL((k_pb_accum<RP, true>), ga, dim3(kPbAccThreads), 0, s, ctx, pb);
      else
        hipLaunchKernelGGL((k_pb_accum<RP, false>), ga, dim3(kPbAccThreads), 0, s, ctx, pb);
      if (pbc.nmulti)
        hipLaunchKernelGGL(k_pb_combine,
                           dim3(grid_for((uint64_t)pbc.nmulti * kPbFineRows, kBlock, 8192)),
                           dim3(kBlock), 0, s, ctx, pb);
    });
    HIP_LAUNCH_CHECK();
    return WL_OK;
  }

  template <typename RP, bool W>
  int spmv_t() {
    const DevState& h = host;
    const bool uniform = !W && h.k == 1 && !ctx.batch;
    if (!W && !uniform && !ctx.batch) {
      bool use = false;
      if (int r = pb_wanted<RP>(&use)) return r;
      if (use) return pb_round<RP>();
    }
    SpmvGrid g;
    g.heavy = h.n_chunks ? grid_for(h.n_chunks, kBlock / kWave) : 0;
    g.b2 = g.heavy + (h.bin_cnt[2] ? grid_for(h.bin_cnt[2], kBlock / 64) : 0);
    g.b1 = g.b2 + (h.bin_cnt[1] ? grid_for(h.bin_cnt[1], kBlock / 16) : 0);
    g.b0 = g.b1 + (h.bin_cnt[0] ? grid_for(h.bin_cnt[0], kBlock / 4) : 0);
    if (g.b0 == 0) return WL_OK;
    const int mode = gather_mode(h.k);
    if (!uniform && mode != kGatherC)
      hipLaunchKernelGGL(k_gather_prep, dim3(grid_for(L.n, kBlock, 4096)), dim3(kBlock),
                         0, s, ctx, mode);
    if (sflags & WL_STATS_WORK)
      hipLaunchKernelGGL(k_count_work<RP>, dim3(grid_for(L.n, kBlock, 4096)),
                         dim3(kBlock), 0, s, ctx, uniform ? kImgUniform : kImgGather, 0);
    timed_spmv(h.round, true, uniform ? kImgUniform : kImgGather, [&] {
      if (uniform)
        hipLaunchKernelGGL(k_spmv_uniform<RP>, dim3(grid_for(L.n, kBlock, 8192)),
                           dim3(kBlock), 0, s, ctx);
      else if (mode == kGather8)
        spmv_launch<RP, W, kGather8>(g);
      else if (mode == kGather16)
        spmv_launch<RP, W, kGather16>(g);
      else
        spmv_launch<RP, W, kGatherC>(g);
    });
    return WL_OK;
  }

  int spmv() {
    if (rp64) return weighted ? spmv_t<uint64_t, true>() : spmv_t<uint64_t, false>();
    return weighted ? spmv_t<uint32_t, true>() : spmv_t<uint32_t, false>();
  }

  // Image of a live round.  The one-colour and propagation-blocking images
  // write z in node order, then loaded into the sort keys; otherwise the
  // rows of the live classes are binned and their images go to the keys
  // directly.
  template <typename RP, bool W>
  int spmv_live_t() {
    const DevState& h = host;
    const bool uniform = !W && h.k == 1 && !ctx.batch;
    const uint32_t gn = grid_for(L.n, kBlock, 4096);
    // right after the one-colour round the member list is the one whose
    // positions that round recorded
    const bool fresh = deg_pos_fresh;
    deg_pos_fresh = false;
    if (!W && !uniform && !ctx.batch) {
      bool use = false;
      if (int r = pb_wanted<RP>(&use)) return r;
      if (use) {
        // then the image goes to the sort keys directly
        pb.kpos = fresh ? ctx.pos_deg : nullptr;
        const int r = pb_round<RP>();
        pb.kpos = nullptr;
        if (r) return r;
        if (!fresh) hipLaunchKernelGGL(k_live_load, dim3(gn), dim3(kBlock), 0, s, ctx);
        return WL_OK;
      }
    }
    if (uniform) {
      if (sflags & WL_STATS_WORK)
        hipLaunchKernelGGL(k_count_work<RP>, dim3(gn), dim3(kBlock), 0, s, ctx, kImgUniform, 1);
      timed_spmv(h.round, true, kImgUniform, [&] {
        hipLaunchKernelGGL(k_spmv_uniform<RP>, dim3(grid_for(L.n, kBlock, 8192)),
                           dim3(kBlock), 0, s, ctx);
      });
      hipLaunchKernelGGL(k_live_load, dim3(gn), dim3(kBlock), 0, s, ctx);
      return WL_OK;
    }
    live_gather<W>(h.round, true);
    return WL_OK;
  }

  int spmv_live() {
    if (rp64) return weighted ? spmv_live_t<uint64_t, true>() : spmv_live_t<uint64_t, false>();
    return weighted ? spmv_live_t<uint32_t, true>() : spmv_live_t<uint32_t, false>();
  }

  // Gathering image of the live rows; every count comes from the device.
  // always: a host-driven round (timed on its own).
  template <bool W>
  void live_gather(uint32_t round, bool always) {
    const uint32_t gl = live_grid();
    if (sflags & WL_STATS_WORK)
      hipLaunchKernelGGL(k_live_count, dim3(gl), dim3(kBlock), 0, s, ctx, 1);
    const uint32_t mid = std::min(live_mid, grid_for(host.nl, kBlock / kWave, 2048));
    const int long_rows = live_heavy || host.max_deg > kShortRow;
    timed_spmv(round, always, kImgGather, [&] {
      // node order (coalesced rows and colours) where the position map is kept:
      // only graphs without long rows keep it
      if (ctx.pos && rp64)
        hipLaunchKernelGGL((k_spmv_node<uint64_t, W>), dim3(grid_for(L.n, kBlock, 4096)),
                           dim3(kBlock), 0, s, ctx);
      else if (ctx.pos)
        hipLaunchKernelGGL((k_spmv_node<uint32_t, W>), dim3(grid_for(L.n, kBlock, 4096)),
                           dim3(kBlock), 0, s, ctx);
      else
        hipLaunchKernelGGL(k_spmv_q<W>, dim3(gl), dim3(kBlock), 0, s, ctx);
      if (live_heavy) {
        const uint32_t gh = grid_for(host.bin_cnt[3], kBlock, 1024);
        hipLaunchKernelGGL(k_heavy_clear, dim3(gh), dim3(kBlock), 0, s, ctx);
        hipLaunchKernelGGL(k_heavy_set, dim3(gh), dim3(kBlock), 0, s, ctx);
      }
      // rows of at most kShortRow entries are done by the first launch alone
      if (long_rows)
        hipLaunchKernelGGL(k_spmv_mid<W>, dim3(live_heavy + mid), dim3(kBlock), 0, s, ctx,
                           live_heavy);
    });
    if (live_heavy)
      hipLaunchKernelGGL(k_live_heavy_fix, dim3(grid_for(host.bin_cnt[3], kBlock, 1024)),
                         dim3(kBlock), 0, s, ctx);
  }

  void spmv_live_async(uint32_t round) {
    if (weighted)
      live_gather<true>(round, false);
    else
      live_gather<false>(round, false);
  }

  // Blocks of k_spmv_mid: the static heavy chunks, then waves for the rows
  // queued per round.
  void plan_live_grid() {
    live_heavy = host.n_chunks ? grid_for(host.n_chunks, kBlock / kWave) : 0;
    live_mid = grid_for(L.n, kBlock / kWave, 2048);
  }

  // Relabel by (c, z) for the current grouping; count_round = 0 for the
  // canonicalisation of the initial labels.
  int relabel(int count_round) {
    if (int r = segmented_sort()) return r;
    relabel_tail(count_round);
    HIP_LAUNCH_CHECK();
    return pull();
  }

  // Sorts the keys inside every class of the current grouping, flags the
  // first position of every distinct (class, key) and ranks the flags
  // (ids, k_new).
  int segmented_sort() {
    const uint32_t gn = grid_for(L.n, kBlock, 4096);
    hipLaunchKernelGGL(k_fill_u8, dim3(gn), dim3(kBlock), 0, s, ctx, ctx.flags,
                       (uint64_t)L.n, (uint8_t)0);
    hipLaunchKernelGGL(k_segments, dim3(grid_for(host.k, kBlock, 4096)), dim3(kBlock),
                       0, s, ctx);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    return finish_sort(0, true);
  }

  // Entries of big-segment list 'which' at the last read-back.
  uint32_t big_entries(int which) const { return (uint32_t)(host.big[which] >> 32); }

  // Radix passes from 'pass0' on while big segments are left (read back after
  // every pass), then the small sorts and, for the full relabel, the rank
  // scan.
  int finish_sort(int pass0, bool full) {
    int pass = pass0;
    for (; pass < kPasses && big_entries(pass & 1) > 0; ++pass) {
      radix_pass(pass, std::min<uint32_t>(big_entries(pass & 1), 4096));
      HIP_LAUNCH_CHECK();
      if (int r = pull()) return r;
    }
    if (pass > pass0) passes_seen = std::max(passes_seen, pass);
    sorts(host.n_tiny ? grid_for(host.n_tiny, kBlock / kWave, 8192) : 0,
          host.n_pico ? grid_for(host.n_pico, kBlock / 8, 8192) : 0,
          std::max<uint32_t>(host.n_msort ? grid_for(host.n_msort, kBlock / kWave, 8192) : 0,
                             std::min<uint32_t>(host.n_small + host.n_msort, 4096)),
          -1);
    if (full) rank_scan();
    HIP_LAUNCH_CHECK();
    return WL_OK;
  }

  void radix_pass(int pass, uint32_t scan_grid) {
    if (pass == 0 && !ctx.keys_mat)
      hipLaunchKernelGGL(k_big_gather, dim3(2048), dim3(kBlock), 0, s, ctx);
    // the first pass of the call clears the histograms over their whole
    // capacity; k_big_scan keeps them cleared after that
    if (!hist_clean) {
      hipLaunchKernelGGL(k_big_clear, dim3(grid_for((uint64_t)L.max_big * kRadix, kBlock, 4096)),
                         dim3(kBlock), 0, s, ctx);
      hist_clean = true;
    }
    hipLaunchKernelGGL(k_big_hist, dim3(1024), dim3(kBlock), 0, s, ctx, pass);
    hipLaunchKernelGGL(k_big_scan, dim3(scan_grid), dim3(kBlock), 0, s, ctx, pass);
    hipLaunchKernelGGL(k_big_scatter, dim3(1024), dim3(kBlock), 0, s, ctx, pass);
    hipLaunchKernelGGL(k_big_copyback, dim3(1024), dim3(kBlock), 0, s, ctx, pass);
  }

  void rank_scan() {
    hipLaunchKernelGGL(k_scan_part, dim3(nscan), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, s, ctx, nscan);
    hipLaunchKernelGGL(k_scan_final, dim3(nscan), dim3(kBlock), 0, s, ctx);
  }

  void relabel_tail(int count_round) {
    const uint32_t gn = grid_for(L.n, kBlock, 4096);
    hipLaunchKernelGGL(k_cstart, dim3(gn), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_scatter_colors, dim3(gn), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_round_end, dim3(1), dim3(1), 0, s, ctx, count_round);
  }

  // Exclusive scan of a (and b) over *lenp entries; totals to tot_a / tot_b.
  // Runs only when *run_if != 0 (run_if NULL: always).
  void xscan(const uint32_t* run_if, const uint32_t* lenp, uint32_t* a, uint32_t* b,
             uint32_t* tot_a, uint32_t* tot_b, uint32_t nblk) {
    hipLaunchKernelGGL(k_xscan_part, dim3(nblk), dim3(kBlock), 0, s, ctx.st, run_if, lenp, a,
                       b, ctx.scan_part);
    hipLaunchKernelGGL(k_xscan_final, dim3(nblk), dim3(kBlock), 0, s, ctx.st, run_if, lenp, a,
                       b, ctx.scan_part, tot_a, tot_b);
  }

  // Live classes from the grouping of the canonical start (perm, cstart, ids
  // = colour of every position, host.k colours).  Once per call.
  int build_live() {
    const uint32_t gn = grid_for(L.n, kBlock, 4096);
    const uint32_t k = host.k;
    DevState* st = ctx.st;
    hipLaunchKernelGGL(k_fill_u8, dim3(grid_for(k, kBlock, 4096)), dim3(kBlock), 0, s, ctx,
                       ctx.gnz, (uint64_t)k, (uint8_t)0);
    if (rp64)
      hipLaunchKernelGGL(k_live_class_nz<uint64_t>, dim3(gn), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_live_class_nz<uint32_t>, dim3(gn), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_live_class_vals, dim3(grid_for(k, kBlock, 4096)), dim3(kBlock), 0, s,
                       ctx);
    xscan(nullptr, &st->k, ctx.gl, ctx.go, &st->n_live2, &st->nl2, nscan);
    if (rp64)
      hipLaunchKernelGGL(k_live_build<uint64_t>, dim3(gn), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_live_build<uint32_t>, dim3(gn), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_live_commit, dim3(gn), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_live_adopt, dim3(1), dim3(1), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    return pull();
  }

  // Sort lists of the live classes.
  void live_segments() {
    hipLaunchKernelGGL(k_live_segments, dim3(grid_for(host.n_live, kBlock, 4096)),
                       dim3(kBlock), 0, s, ctx);
  }

  // Grids of the kernels over the live positions: sized from the last count
  // read back (the live set only shrinks, so it bounds every later round).
  uint32_t live_grid() const { return grid_for(host.nl, kBlock, 4096); }
  uint32_t live_scan_blocks() const { return scan_blocks(host.nl); }

  // After the sort: sub-classes, new colours of every node, next live
  // classes, end of the round.
  // async: a device-driven round, which launches no kernels for the
  // per-colour shift table; a round that needs the table halts the device in
  // k_shift_apply (finish_halted builds it).
  void live_tail(bool async = false) {
    const uint32_t gl = live_grid(), ns = live_scan_blocks();
    const uint32_t gc = grid_for(host.n_live, kBlock, 4096);
    DevState* st = ctx.st;
    hipLaunchKernelGGL(k_live_scan_part, dim3(ns), dim3(kBlock), 0, s, ctx);
    if (rp64)
      hipLaunchKernelGGL(k_live_scan_final<uint64_t>, dim3(ns), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_live_scan_final<uint32_t>, dim3(ns), dim3(kBlock), 0, s, ctx);
    // its first ns blocks leave the block sums of the scan of gl and go
    hipLaunchKernelGGL(k_live_subs_splits, dim3(std::max(std::max(gl, gc), ns)), dim3(kBlock), 0,
                       s, ctx, ns);
    hipLaunchKernelGGL(k_xscan_final, dim3(ns), dim3(kBlock), 0, s, ctx.st, &st->split_any,
                       &st->nsub, ctx.gl, ctx.go, ctx.scan_part, &st->n_live2, &st->nl2);
    live_shift_end(!async);
  }

  // The per-colour shift table (when with_table; it is built only if the
  // round's splits need it), the new colour of every node, the next live
  // classes and the end of the round.
  void live_shift_end(bool with_table) {
    const uint32_t gn = grid_for(L.n, kBlock, 4096);
    const uint32_t gl = live_grid();
    const uint32_t gc = grid_for(host.n_live, kBlock, 4096);
    DevState* st = ctx.st;
    if (with_table) {
      hipLaunchKernelGGL(k_shift_clear, dim3(gn), dim3(kBlock), 0, s, ctx);
      hipLaunchKernelGGL(k_shift_scatter, dim3(gc), dim3(kBlock), 0, s, ctx);
      xscan(&st->shift_big, &st->k, ctx.shift, nullptr, nullptr, nullptr, nscan);
    }
    // each block loads the split list into LDS: a capped grid loads it fewer times
    hipLaunchKernelGGL(k_shift_apply, dim3(std::min<uint32_t>(gn, 1024)), dim3(kBlock), 0, s,
                       ctx, with_table ? 0 : 1);
    if (rp64)
      hipLaunchKernelGGL(k_live_emit<uint64_t>, dim3(gl), dim3(kBlock), 0, s, ctx);
    else
      hipLaunchKernelGGL(k_live_emit<uint32_t>, dim3(gl), dim3(kBlock), 0, s, ctx);
    hipLaunchKernelGGL(k_live_round_end, dim3(1), dim3(1), 0, s, ctx);
  }

  // The one-colour round of an unweighted graph without a sort
  // (wl_degree.h).  *handled is false when the graph has more distinct
  // degrees than one workgroup ranks; the caller then runs the general round.
  template <bool RP64>
  int degree_round(bool* handled) {
    *handled = false;
    const uint32_t maxd = host.max_deg;
    DegScratch d;
    uint32_t* base = (uint32_t*)ctx.keys_tmp;
    d.dcount = base;
    d.dlist = base + (uint64_t)maxd + 1;
    d.roff = d.dlist + kDegRanks;
    d.rj = d.roff + kDegRanks;
    d.rdeg = d.rj + kDegRanks;
    d.nd = &ctx.st->deg_nd;
    const uint32_t gd = grid_for((uint64_t)maxd + 1, kBlock, 4096);
    using RPT = typename std::conditional<RP64, uint64_t, uint32_t>::type;
    if (sflags & WL_STATS_WORK)
      hipLaunchKernelGGL(k_count_work<RPT>, dim3(grid_for(L.n, kBlock, 4096)), dim3(kBlock), 0,
                         s, ctx, kImgUniform, 1);
    timed_spmv(host.round, true, kImgUniform, [&] {
      hipLaunchKernelGGL(k_deg_clear, dim3(gd), dim3(kBlock), 0, s, ctx, d, maxd);
      hipLaunchKernelGGL(k_deg_hist<RP64>, dim3(grid_for(L.n, kBlock, 4096)), dim3(kBlock), 0,
                         s, ctx, d);
    });
    hipLaunchKernelGGL(k_deg_list, dim3(gd), dim3(kBlock), 0, s, ctx, d, maxd);
    hipLaunchKernelGGL(k_deg_ranks, dim3(1), dim3(kDegThreads), 0, s, ctx, d);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    if (host.deg_nd > kDegRanks) return WL_OK;
    // the rank x block matrix of the placement lives in x (2n words): at
    // most 1024 blocks, fewer when there are many ranks
    const uint64_t K = std::max<uint32_t>(host.k_new, 1);
    const uint32_t nblk = (uint32_t)std::max<uint64_t>(
        1, std::min<uint64_t>({1024, grid_for(L.n, kBlock), 2 * L.n / K}));
    uint32_t* m = (uint32_t*)ctx.x;
    hipLaunchKernelGGL(k_deg_count<RP64>, dim3(nblk), dim3(kBlock), 0, s, ctx, d, m);
    hipLaunchKernelGGL(k_deg_rowscan, dim3((uint32_t)std::min<uint64_t>(K, 4096)), dim3(kBlock), 0,
                       s, ctx, d, m, nblk);
    hipLaunchKernelGGL(k_deg_fill, dim3(grid_for((uint64_t)L.n / 4 + 1, kBlock, 1024)),
                       dim3(kBlock), 0, s, ctx, d);
    hipLaunchKernelGGL(k_deg_place<RP64>, dim3(nblk), dim3(kBlock), 0, s, ctx, d, m);
    hipLaunchKernelGGL(k_live_round_end, dim3(1), dim3(1), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    *handled = true;
    deg_pos_fresh = ctx.pos_deg != nullptr && !host.done;
    return WL_OK;
  }

  // Whether the degree round's table and lists fit the scratch it uses (the
  // keys_tmp region, two words per node).
  bool degree_round_fits() const {
    const uint64_t words = (uint64_t)host.max_deg + 1 + 4ull * kDegRanks;
    return host.max_deg < 0x7FFFFFFFu && words <= 2 * L.n;
  }

  // One round of the incremental relabel driven from the host (counts read
  // back to size the sorts).
  bool degree_round_applies() const {
    return host.k == 1 && !weighted && !ctx.batch && deg_mode && degree_round_fits();
  }

  void use_round_ctx(uint32_t round) {
    ctx = ((round - live_r0) & 1) ? swapped_live(ctx0) : ctx0;
  }

  // Builds the live classes into buffer set 0 for the coming round, whose
  // counters it also sets.
  int build_live_now() {
    ctx = ctx0;
    if (int r = build_live()) return r;
    live_built = true;
    live_r0 = host.round;
    hipLaunchKernelGGL(k_round_begin, dim3(1), dim3(1), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    return WL_OK;
  }

  // Live positions from which a host-driven round launches its first two
  // radix passes before reading anything back.
  static constexpr uint32_t kBlindPassesMin = 1u << 20;

  int round_live() {
    if (degree_round_applies()) {
      ctx = ctx0;
      hipLaunchKernelGGL(k_round_begin, dim3(1), dim3(1), 0, s, ctx);
      bool handled = false;
      if (int r = rp64 ? degree_round<true>(&handled) : degree_round<false>(&handled)) return r;
      if (handled) {
        live_built = true;
        live_r0 = host.round;
        return WL_OK;
      }
    }
    if (!live_built)
      if (int r = build_live_now()) return r;
    use_round_ctx(host.round);
    hipLaunchKernelGGL(k_round_begin, dim3(1), dim3(1), 0, s, ctx);
    if (int r = spmv_live()) return r;
    live_segments();
    if (host.nl >= kBlindPassesMin) {
      // a large live set: the first two radix passes go out without a
      // read-back (a pass whose list is empty returns at once); the
      // read-back after them sizes the small sorts and shows whether more
      // passes are needed.  Pass 1 had work when pass 0 left big buckets.
      radix_pass(0, 1024);
      radix_pass(1, 1024);
      HIP_LAUNCH_CHECK();
      if (int r = pull()) return r;
      passes_seen = std::max(passes_seen, big_entries(1) > 0 ? 2 : 1);
      if (int r = finish_sort(2, false)) return r;
    } else {
      HIP_LAUNCH_CHECK();
      if (int r = pull()) return r;
      if (int r = finish_sort(0, false)) return r;
    }
    live_tail();
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    if (host.err & kErrNotSymmetric)
      return fail(WL_EINVAL, "the graph is flagged symmetric but is not");
    if (host.err & kErrChain) return fail(WL_EHIP, "a chained scan did not complete");
    return WL_OK;
  }

  // Radix passes launched per device-driven round: as many as the rounds so
  // far needed (at least one), at most async_passes.
  int async_pass_count() const {
    return std::min(async_passes, std::max(1, passes_seen));
  }

  // The same launched without reading anything back: grids are fixed for the
  // call and counts come from the device state; the per-round counters were
  // set by the previous round's end.  A round that needs
  // more radix passes than it launches halts the device before its small
  // sorts (finish_halted completes it).
  void round_live_async(uint32_t round) {
    use_round_ctx(round);
    spmv_live_async(round);
    live_segments();
    const int ap = async_pass_count();
    for (int pass = 0; pass < ap; ++pass) radix_pass(pass, 1024);
    // the small sorts' grids: enough blocks to fill the device, the segments
    // taken in grid-stride loops
    sorts(grid_for(L.n / 2, kBlock / kWave, 1024), grid_for(L.n / 2, kBlock / 8, 1024),
          grid_for(L.n / (kTinyMax + 1), 1, 1024), ap);
    live_tail(true);
  }

  // The graph of rounds r, r + 1 for a first round of parity p = (r -
  // live_r0) & 1, (re)captured when the radix pass count changed.  The
  // grids are those of the capture; the live set only shrinks, so they stay
  // large enough.
  int ensure_graph(int p, uint32_t r) {
    const int ap = async_pass_count();
    if (gexec[p] && gexec_ap[p] == ap) return WL_OK;
    if (gexec[p]) {
      HIP_TRY(hipGraphExecDestroy(gexec[p]));
      gexec[p] = nullptr;
    }
    if (!cap_stream) HIP_TRY(hipStreamCreateWithFlags(&cap_stream, hipStreamNonBlocking));
    const hipStream_t s0 = s;
    s = cap_stream;
    capturing = true;
    hipGraph_t g = nullptr;
    hipError_t e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
    if (e == hipSuccess) {
      round_live_async(r);
      round_live_async(r + 1);
      e = hipStreamEndCapture(s, &g);
    }
    s = s0;
    capturing = false;
    if (e != hipSuccess)
      return fail(WL_EHIP, "graph capture of the rounds failed: %s", hipGetErrorString(e));
    e = hipGraphInstantiate(&gexec[p], g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) {
      gexec[p] = nullptr;
      return fail(WL_EHIP, "graph instantiation failed: %s", hipGetErrorString(e));
    }
    gexec_ap[p] = ap;
    return WL_OK;
  }

  // Queues rounds base .. base + count - 1 (count even) without a read-back.
  int launch_async_rounds(uint32_t base, uint32_t count) {
    if (!use_graph) {
      for (uint32_t i = 0; i < count; ++i) round_live_async(base + i);
      HIP_LAUNCH_CHECK();
      return WL_OK;
    }
    const int p = (int)((base - live_r0) & 1);
    if (int r = ensure_graph(p, base)) return r;
    for (uint32_t i = 0; i < count; i += 2) HIP_TRY(hipGraphLaunch(gexec[p], s));
    // each replayed round has one gathering image launch: counted when the
    // round ran, without a time
    for (uint32_t i = 0; i < count; ++i)
      timed.push_back(TimedSpmv{nullptr, nullptr, base + i, false, kImgGather});
    return WL_OK;
  }

  // The device halted in a round, after async_passes radix passes
  // (kHalted) or before the shift table (kHaltedShift): clear the halt and
  // finish that round from there, host-driven.
  int finish_halted() {
    const uint32_t why = host.done;
    use_round_ctx(host.round);
    hipLaunchKernelGGL(k_resume, dim3(1), dim3(1), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    if (why == kHaltedShift) {
      live_shift_end(true);
    } else {
      if (int r = finish_sort(async_pass_count(), false)) return r;
      live_tail();
    }
    HIP_LAUNCH_CHECK();
    return pull();
  }

  // Algorithm 1 to completion on the session's graph, from labels on the
  // device (or the trivial partition).  Leaves colours in ctx.c.
  int run_rsc(const uint32_t* init_dev) {
    const uint32_t gn = grid_for(L.n, kBlock, 4096);
    hipLaunchKernelGGL(k_iota_zero, dim3(gn), dim3(kBlock), 0, s, ctx);
    HIP_LAUNCH_CHECK();
    if (init_dev) {
      hipLaunchKernelGGL(k_labels_to_z, dim3(gn), dim3(kBlock), 0, s, ctx, init_dev);
      HIP_LAUNCH_CHECK();
      if (int r = relabel(0)) return r;
    }
    if (int r = build_schedule(true)) return r;
    ctx.keys_mat = 1;
    // The live rows are gathered in node order only when every row is short:
    // with long rows, node order puts rows of very different lengths in one
    // wave, while the class order groups rows of equal length.
    if (host.max_deg > kShortRow) ctx.pos = nullptr;
    ctx0 = ctx;
    // The live classes come from the grouping above, unless the first round
    // is the one-colour degree round, which builds them itself.
    if (!degree_round_applies())
      if (int r = build_live_now()) return r;
    live_mode = true;
    plan_live_grid();
    // The first rounds are driven from the host (each reads its counts
    // back); after that, rounds go to the device in groups of 'ahead' with
    // one read-back per group.  Rounds queued past the last one find the
    // state done and return at once.
    uint32_t host_rounds = 0, ahead = 8;
    while (!host.done) {
      if (host_rounds < host_rounds_first) {
        if (int r = round_live()) return r;
        ++host_rounds;
        continue;
      }
      if (!live_built)
        if (int r = build_live_now()) return r;
      if (int r = launch_async_rounds(host.round, ahead)) return r;
      if (int r = pull()) return r;
      if (host.done == kHalted || host.done == kHaltedShift)
        if (int r = finish_halted()) return r;
      if (host.err & kErrNotSymmetric)
        return fail(WL_EINVAL, "the graph is flagged symmetric but is not");
      if (host.err & kErrChain) return fail(WL_EHIP, "a chained scan did not complete");
      ahead = std::min<uint32_t>(ahead * 2, 64);
    }
    return WL_OK;
  }

  int round() {
    hipLaunchKernelGGL(k_round_begin, dim3(1), dim3(1), 0, s, ctx);
    if (int r = spmv()) return r;
    HIP_LAUNCH_CHECK();
    if (int r = relabel(1)) return r;
    if (host.err & kErrNotSymmetric)
      return fail(WL_EINVAL, "the graph is flagged symmetric but is not");
    return WL_OK;
  }
};

int open_session(Session& S, const wl_csr* g, uint32_t* colors, void* ws,
                 uint64_t ws_bytes, void* stream, bool in_core = true) {
  S.L = make_layout(g->n, g->nnz, in_core);
  if (!ws) return fail(WL_EINVAL, "workspace is NULL");
  if ((uintptr_t)ws % kAlign)
    return fail(WL_EINVAL, "workspace must be %llu-byte aligned",
                (unsigned long long)kAlign);
  if (ws_bytes < S.L.total)
    return fail(WL_EBUDGET, "workspace has %llu bytes, %llu needed",
                (unsigned long long)ws_bytes, (unsigned long long)S.L.total);
  S.ctx = make_ctx(S.L, g, (uint8_t*)ws, colors);
  S.s = (hipStream_t)stream;
  S.rp64 = g->row_ptr64 != nullptr;
  S.weighted = g->weight != nullptr;
  S.nscan = scan_blocks(g->n);
  S.host_rounds_first = (uint32_t)env_int("WL_HOST_ROUNDS", 0, 1 << 30, (int)kHostRounds);
  S.async_passes = env_int("WL_ASYNC_PASSES", 0, kPasses, kAsyncPassesDefault);
  {
    const char* m = getenv("WL_PB");
    S.pb_mode = !m ? 1 : (strcmp(m, "0") == 0 ? 0 : (strcmp(m, "force") == 0 ? 2 : 1));
  }
  S.sym_flag = (g->flags & WL_CSR_SYMMETRIC) != 0;
  S.deg_mode = env_int("WL_DEGREE_ROUND", 0, 1, 1) != 0;
  S.use_graph = env_int("WL_GRAPH", 0, 1, 0) != 0;
  if (wants_pb(g) && S.pb_mode != 0) {
    S.P = make_pb_layout(g->n, g->nnz);
    // pass 1 reads the column indices 16 bytes at a time
    if (S.P.ok && ws_bytes >= S.L.total + S.P.total && (uintptr_t)g->col_idx % 16 == 0) {
      uint8_t* B = (uint8_t*)ws + S.L.total;
      PbCtx& p = S.pb;
      p.levels = S.P.levels;
      p.shift1 = S.P.shift1;
      p.nb1 = S.P.nb1;
      p.nfine = S.P.nfine;
      p.fbits = S.P.fbits;
      p.ntiles1 = S.P.ntiles1;
      p.cnt = (PbCounts*)(B + S.P.cnt);
      p.bstart1 = (uint64_t*)(B + S.P.bstart1);
      p.bstartf = (uint64_t*)(B + S.P.bstartf);
      p.rec1 = (uint32_t*)(B + S.P.rec1);
      p.rec2 = (uint32_t*)(B + S.P.rec2);
      p.tile_row = (uint32_t*)(B + S.P.tile_row);
      p.tile2_off = (uint32_t*)(B + S.P.tile2_off);
      p.cur1 = (unsigned long long*)(B + S.P.cur1);
      p.cur2 = (unsigned long long*)(B + S.P.cur2);
      p.slice_off = (uint32_t*)(B + S.P.slice_off);
      p.mslice_off = (uint32_t*)(B + S.P.mslice_off);
      p.mlist = (uint32_t*)(B + S.P.mlist);
      p.part = (uint64_t*)(B + S.P.part);
      S.pb_avail = true;
    }
  }
  return WL_OK;
}

#include "wl_outofcore.h"

// ---------------------------------------------------------------------------
// Exact stability certificate (Definition "Stable Coloring").
// ---------------------------------------------------------------------------

struct VerLayout {
  uint64_t st, rep, multi, mid, hub, hub_off, keys, total;
};

VerLayout ver_layout(uint64_t n, uint64_t nnz, bool weighted) {
  VerLayout L{};
  uint64_t o = 0;
  auto take = [&](uint64_t b) { uint64_t at = o; o = align_up(o + b); return at; };
  L.st = take(sizeof(VerState));
  L.rep = take(4 * n);
  L.multi = take(n);
  L.mid = take(4 * n);
  L.hub = take(4 * n);
  L.hub_off = take(4 * (n + 1));
  L.keys = take((weighted ? 8 : 4) * nnz);
  L.total = o;
  return L;
}

template <typename K>
int verify_run(const wl_csr* g, const uint32_t* color, uint32_t k, uint8_t* ws,
               const VerLayout& L, hipStream_t s) {
  VerCtx<K> v{};
  v.n = (uint32_t)g->n;
  v.k = k;
  v.rp32 = g->row_ptr32;
  v.rp64 = g->row_ptr64;
  v.col = g->col_idx;
  v.wgt = g->weight;
  v.color = color;
  v.st = (VerState*)(ws + L.st);
  v.rep = (uint32_t*)(ws + L.rep);
  v.multi = ws + L.multi;
  v.mid = (uint32_t*)(ws + L.mid);
  v.hub = (uint32_t*)(ws + L.hub);
  v.hub_off = (uint32_t*)(ws + L.hub_off);
  v.keys = (K*)(ws + L.keys);
  VerState h{};
  auto pull = [&]() -> int {
    HIP_TRY(hipMemcpyAsync(&h, v.st, sizeof(VerState), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return WL_OK;
  };
  const uint32_t gn = grid_for(v.n, kBlock, 4096);
  hipLaunchKernelGGL(k_v_clear<K>, dim3(grid_for(k, kBlock, 4096)), dim3(kBlock), 0, s, v);
  hipLaunchKernelGGL(k_v_rep<K>, dim3(gn), dim3(kBlock), 0, s, v);
  HIP_LAUNCH_CHECK();
  if (int r = pull()) return r;
  if (h.err & kVErrColor) return fail(WL_EINVAL, "a colour is >= k");
  hipLaunchKernelGGL(k_v_multi<K>, dim3(gn), dim3(kBlock), 0, s, v);
  hipLaunchKernelGGL(k_v_bin<K>, dim3(gn), dim3(kBlock), 0, s, v);
  hipLaunchKernelGGL(k_v_sort_wave<K>, dim3(grid_for(v.n, kBlock / kWave, 8192)),
                     dim3(kBlock), 0, s, v);
  HIP_LAUNCH_CHECK();
  if (int r = pull()) return r;
  if (h.n_mid)
    hipLaunchKernelGGL(k_v_sort_mid<K>, dim3(std::min<uint32_t>(h.n_mid, 4096)),
                       dim3(kBlock), 0, s, v);
  if (h.n_hub) {
    hipLaunchKernelGGL(k_v_hub_plan<K>, dim3(1), dim3(kBlock), 0, s, v);
    HIP_LAUNCH_CHECK();
    if (int r = pull()) return r;
    const uint32_t gc = std::min<uint32_t>(h.n_hub_chunks, 8192);
    hipLaunchKernelGGL(k_v_hub_sort_chunks<K>, dim3(gc), dim3(kBlock), 0, s, v);
    for (uint64_t kk = 2ull * kVChunk; kk <= h.max_pow; kk <<= 1) {
      hipLaunchKernelGGL(k_v_hub_step<K>, dim3(gc), dim3(kBlock), 0, s, v, kk, kk, 1);
      for (uint64_t j = kk >> 2; j >= kVChunk; j >>= 1)
        hipLaunchKernelGGL(k_v_hub_step<K>, dim3(gc), dim3(kBlock), 0, s, v, kk, j, 0);
      hipLaunchKernelGGL(k_v_hub_finish<K>, dim3(gc), dim3(kBlock), 0, s, v, kk);
    }
  }
  if constexpr (sizeof(K) == 4)
    hipLaunchKernelGGL(k_v_compare, dim3(grid_for(v.n, kBlock / 16, 8192)), dim3(kBlock), 0,
                       s, v);
  else
    hipLaunchKernelGGL(k_v_compare_w, dim3(gn), dim3(kBlock), 0, s, v);
  HIP_LAUNCH_CHECK();
  if (int r = pull()) return r;
  return (h.err & kVErrMismatch) ? fail(WL_ENOTSTABLE, "the colouring is not stable") : WL_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

// Device scratch of wl_stable_coloring_noalloc: one array per GPU, held for
// the life of the process, in place of the caller's workspace.  Host code
// never passes 'scratch' itself to a kernel or a copy: its device address on
// the current GPU comes from hipGetSymbolAddress (scratch_address below).
__device__ __align__(256) uint8_t scratch[WL_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of 'scratch' on the current device, looked up once per
// device and kept.
int scratch_address(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(WL_EINVAL, "device %d is beyond the %d devices the scratch table holds", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(WL_EHIP, "hipGetSymbolAddress gave no address for the scratch");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return WL_OK;
}
}  // namespace

extern "C" {

const char* wl_last_error(void) { return g_err; }

int wl_set_precision(uint32_t q) {
  g_err[0] = 0;
  if (q != WL_PRECISION_FP && q != WL_PRECISION_RING64)
    return fail(WL_EINVAL, "precision %u: use 0 (F_p) or 64 (Z/2^64)", q);
  g_ring = q == WL_PRECISION_RING64 ? 1u : 0u;
  return WL_OK;
}

int wl_get_precision(uint32_t* q) {
  g_err[0] = 0;
  if (!q) return fail(WL_EINVAL, "NULL argument");
  *q = g_ring ? WL_PRECISION_RING64 : WL_PRECISION_FP;
  return WL_OK;
}

int wl_stats_enable(int flags) {
  if (flags & ~(WL_STATS_TIME | WL_STATS_WORK)) return fail(WL_EINVAL, "unknown flag");
  g_stats_flags = flags;
  return WL_OK;
}

int wl_stats_get(wl_stats* out) {
  if (!out) return fail(WL_EINVAL, "NULL argument");
  *out = g_stats;
  return WL_OK;
}

int wl_workspace_size(const wl_csr* g, uint64_t* bytes_out) {
  g_err[0] = 0;
  if (!g || !bytes_out) return fail(WL_EINVAL, "NULL argument");
  if (g->n >= (1ull << 32)) return fail(WL_EOVERFLOW, "n does not fit 32 bits");
  uint64_t bytes = make_layout(g->n, g->nnz).total;
  if (wants_pb(g)) {
    const PbLayout P = make_pb_layout(g->n, g->nnz);
    if (P.ok) bytes += P.total;
  }
  *bytes_out = bytes;
  return WL_OK;
}

int wl_batched_workspace_size(const wl_csr* g, uint64_t max_batch_entries,
                              uint64_t* bytes_out) {
  g_err[0] = 0;
  if (!g || !bytes_out) return fail(WL_EINVAL, "NULL argument");
  if (g->n >= (1ull << kQShift))
    return fail(WL_EOVERFLOW, "the batched path needs n < 2^%d", kQShift);
  const uint64_t mb = max_batch_entries ? max_batch_entries : std::max<uint64_t>(g->nnz, 1);
  *bytes_out = std::max(refine_layout(g->n, mb).total, quot_layout(g->n, 1).total);
  return WL_OK;
}

int wl_refine_round(const wl_csr* g, const uint32_t* color_in, uint32_t k_in,
                    uint64_t seed, uint32_t round, uint32_t* color_out,
                    uint32_t* k_out, void* workspace, uint64_t ws_bytes,
                    void* stream) {
  g_err[0] = 0;
  if (int r = check_graph(g)) return r;
  if (!k_out) return fail(WL_EINVAL, "k_out is NULL");
  if (g->n == 0) {
    *k_out = 0;
    return WL_OK;
  }
  if (!color_in || !color_out) return fail(WL_EINVAL, "colour buffer is NULL");
  if (k_in == 0 || k_in > g->n)
    return fail(WL_EINVAL, "k_in = %u must be in [1, n]", k_in);
  Session S;
  if (int r = open_session(S, g, color_out, workspace, ws_bytes, stream)) return r;
  if (int r = check_nnz_device(g, S.s)) return r;
  if (int r = S.init_state(seed, k_in, round, round + 1, 0)) return r;
  if (int r = S.validate_device()) return r;
  if (int r = S.check_ring()) return r;
  const uint32_t gn = grid_for(g->n, kBlock, 4096);
  hipLaunchKernelGGL(k_check_colors, dim3(gn), dim3(kBlock), 0, S.s, S.ctx, color_in,
                     k_in);
  HIP_LAUNCH_CHECK();
  if (int r = S.pull()) return r;
  if (S.host.err & 4u) return fail(WL_EINVAL, "a colour is >= k_in");
  if (color_out != color_in)
    HIP_TRY(hipMemcpyAsync(color_out, color_in, 4 * g->n, hipMemcpyDeviceToDevice, S.s));
  hipLaunchKernelGGL(k_count_colors, dim3(grid_for(k_in + 1)), dim3(kBlock), 0, S.s,
                     S.ctx, k_in);
  hipLaunchKernelGGL(k_hist_colors, dim3(gn), dim3(kBlock), 0, S.s, S.ctx);
  hipLaunchKernelGGL(k_scan_colors, dim3(1), dim3(kBlock), 0, S.s, S.ctx, k_in);
  hipLaunchKernelGGL(k_place_colors, dim3(gn), dim3(kBlock), 0, S.s, S.ctx);
  HIP_LAUNCH_CHECK();
  if (int r = S.stats_begin()) return r;
  if (int r = S.build_schedule()) return r;
  if (int r = S.round()) return r;
  if (int r = S.stats_end()) return r;
  *k_out = S.host.k;
  return WL_OK;
}

int wl_stable_coloring(const wl_csr* g, const uint32_t* init_color, uint64_t seed,
                       uint32_t max_rounds, uint32_t* color_out, uint32_t* k_out,
                       uint32_t* rounds_out, void* workspace, uint64_t ws_bytes,
                       void* stream) {
  g_err[0] = 0;
  if (int r = check_graph(g)) return r;
  if (!k_out || !rounds_out) return fail(WL_EINVAL, "output scalar is NULL");
  *k_out = 0;
  *rounds_out = 0;
  if (g->n == 0) return WL_OK;
  if (!color_out) return fail(WL_EINVAL, "color_out is NULL");
  Session S;
  if (int r = open_session(S, g, color_out, workspace, ws_bytes, stream)) return r;
  if (int r = check_nnz_device(g, S.s)) return r;
  const uint32_t cap = max_rounds ? max_rounds : (uint32_t)std::min<uint64_t>(g->n + 1, 0xFFFFFFFFull);
  if (int r = S.init_state(seed, 1, 0, cap, 1)) return r;
  if (int r = S.validate_device()) return r;
  if (int r = S.check_ring()) return r;
  if (int r = S.stats_begin()) return r;
  if (int r = S.run_rsc(init_color)) return r;
  if (int r = S.stats_end()) return r;
  *k_out = S.host.k;
  *rounds_out = S.host.round;
  if (S.host.done == 2)
    return fail(WL_EMAXROUNDS, "no stable colouring after %u rounds", S.host.round);
  return WL_OK;
}

int wl_stable_coloring_noalloc(const wl_csr* g, const uint32_t* init_color, uint64_t seed,
                               uint32_t max_rounds, uint32_t* color_out, uint32_t* k_out,
                               uint32_t* rounds_out, void* stream) {
  g_err[0] = 0;
  if (int r = check_graph(g)) return r;
  if (!k_out || !rounds_out) return fail(WL_EINVAL, "output scalar is NULL");
  *k_out = 0;
  *rounds_out = 0;
  if (g->n == 0) return WL_OK;
  if (!color_out) return fail(WL_EINVAL, "color_out is NULL");
  // the in-core layout must fit the scratch (the binned image is used only
  // when its larger layout fits as well)
  const uint64_t need = make_layout(g->n, g->nnz).total;
  if (need > WL_NOALLOC_SCRATCH_BYTES)
    return fail(WL_EBUDGET,
                "graph needs %llu bytes of workspace; the fixed scratch holds %llu "
                "(use wl_stable_coloring with a workspace of that size)",
                (unsigned long long)need, (unsigned long long)WL_NOALLOC_SCRATCH_BYTES);
  if (stream) {
    int sdev = -1, cur = -1;
    HIP_TRY(hipStreamGetDevice((hipStream_t)stream, &sdev));
    HIP_TRY(hipGetDevice(&cur));
    if (sdev != cur)
      return fail(WL_EINVAL, "the stream belongs to device %d, the current device is %d",
                  sdev, cur);
  }
  void* ws = nullptr;
  if (int r = scratch_address(&ws)) return r;
  Session S;
  if (int r = open_session(S, g, color_out, ws, WL_NOALLOC_SCRATCH_BYTES, stream)) return r;
  S.use_graph = false;  // no graph objects: nothing is created
  if (int r = check_nnz_device(g, S.s)) return r;
  const uint32_t cap = max_rounds ? max_rounds : (uint32_t)std::min<uint64_t>(g->n + 1, 0xFFFFFFFFull);
  if (int r = S.init_state(seed, 1, 0, cap, 1)) return r;
  if (int r = S.validate_device()) return r;
  if (int r = S.check_ring()) return r;
  if (int r = S.run_rsc(init_color)) return r;
  if (int r = S.pull()) return r;
  *k_out = S.host.k;
  *rounds_out = S.host.round;
  if (S.host.done == 2)
    return fail(WL_EMAXROUNDS, "no stable colouring after %u rounds", S.host.round);
  return WL_OK;
}

int wl_stable_coloring_batched(const wl_csr* g_host, const uint32_t* init_host,
                               uint64_t seed, uint64_t max_batch_entries, uint32_t options,
                               uint32_t* color_out_host, uint32_t* k_out,
                               uint32_t* rounds_out, uint32_t* outer_out,
                               int* coarsest_out, void* workspace, uint64_t ws_bytes,
                               void* stream) {
  g_err[0] = 0;
  if (int r = check_graph(g_host)) return r;
  if (!k_out || !rounds_out || !outer_out || !coarsest_out)
    return fail(WL_EINVAL, "output scalar is NULL");
  *k_out = 0;
  *rounds_out = 0;
  *outer_out = 0;
  *coarsest_out = 1;
  if (g_host->n >= (1ull << kQShift))
    return fail(WL_EOVERFLOW, "the batched path needs n < 2^%d", kQShift);
  if (g_host->n == 0) return WL_OK;
  if (!color_out_host) return fail(WL_EINVAL, "color_out_host is NULL");
  if (!workspace) return fail(WL_EINVAL, "workspace is NULL");
  if ((uintptr_t)workspace % kAlign) return fail(WL_EINVAL, "workspace must be 256-byte aligned");
  const uint64_t last = g_host->row_ptr64 ? g_host->row_ptr64[g_host->n]
                                          : g_host->row_ptr32[g_host->n];
  if (last != g_host->nnz) return fail(WL_EINVAL, "row_ptr[n] != nnz");
  if (options & ~(WL_BATCHED_EXACT | WL_BATCHED_EARLY_STOP))
    return fail(WL_EINVAL, "unknown option bits 0x%x", options);
  // The exact finish is enabled only up to the largest graph it has been
  // verified on; above it, one run ended in a host fault whose cause is not
  // known (a quotient of 1.7e10 weighted entries in pageable memory).
  if ((options & WL_BATCHED_EXACT) && g_host->nnz > kExactFinishMaxEntries)
    return fail(WL_EINVAL,
                "WL_BATCHED_EXACT is limited to graphs of at most 2^31 entries (%llu given); "
                "use wl_stable_coloring_streamed for the exact colouring of a larger graph",
                (unsigned long long)g_host->nnz);
  if (g_ring) {
    // a quotient row sums the entries of its representative's row, so the
    // input's bound holds for every quotient
    HostGraph G;
    G.n = g_host->n;
    G.m = g_host->nnz;
    G.rp32 = g_host->row_ptr32;
    G.rp64 = g_host->row_ptr64;
    G.wt = g_host->weight;
    HostPool pool;
    if (!ring_row_sums_ok(pool, G))
      return fail(WL_EOVERFLOW, "a row sum exceeds 2^32, the bound of arithmetic mod 2^64");
  }
  return batched_run(g_host, init_host, seed, max_batch_entries, options, color_out_host, k_out,
                     rounds_out, outer_out, coarsest_out, workspace, ws_bytes,
                     (hipStream_t)stream);
}

int wl_streamed_workspace_size(const wl_csr* g, uint64_t* bytes_out) {
  g_err[0] = 0;
  if (!g || !bytes_out) return fail(WL_EINVAL, "NULL argument");
  if (g->n >= (1ull << 31)) return fail(WL_EOVERFLOW, "the streamed path needs n < 2^31");
  HostGraph G;
  G.n = g->n;
  G.m = g->nnz;
  *bytes_out = stream_layout(g->n, stream_chunk_cap(G), g->weight != nullptr).total;
  return WL_OK;
}

int wl_stable_coloring_streamed(const wl_csr* g_host, const uint32_t* init_host, uint64_t seed,
                                uint32_t max_rounds, uint32_t* color_out_host, uint32_t* k_out,
                                uint32_t* rounds_out, void* workspace, uint64_t ws_bytes,
                                void* stream) {
  g_err[0] = 0;
  if (int r = check_graph(g_host)) return r;
  if (!k_out || !rounds_out) return fail(WL_EINVAL, "output scalar is NULL");
  *k_out = 0;
  *rounds_out = 0;
  if (g_host->n >= (1ull << 31)) return fail(WL_EOVERFLOW, "the streamed path needs n < 2^31");
  if (g_host->n == 0) return WL_OK;
  if (!color_out_host) return fail(WL_EINVAL, "color_out_host is NULL");
  if (!workspace) return fail(WL_EINVAL, "workspace is NULL");
  if ((uintptr_t)workspace % kAlign) return fail(WL_EINVAL, "workspace must be 256-byte aligned");
  HostGraph G;
  G.n = g_host->n;
  G.m = g_host->nnz;
  G.rp32 = g_host->row_ptr32;
  G.rp64 = g_host->row_ptr64;
  G.col = g_host->col_idx;
  G.wt = g_host->weight;
  if (G.rp(0) != 0 || G.rp(G.n) != G.m) return fail(WL_EINVAL, "row_ptr[0] != 0 or row_ptr[n] != nnz");
  for (uint64_t i = 0; i < G.n; ++i)
    if (G.rp(i + 1) < G.rp(i)) return fail(WL_EINVAL, "row_ptr is not non-decreasing");
  if (G.m > 0 && !G.col) return fail(WL_EINVAL, "col_idx is NULL");
  if (g_ring) {
    HostPool pool;
    if (!ring_row_sums_ok(pool, G))
      return fail(WL_EOVERFLOW, "a row sum exceeds 2^32, the bound of arithmetic mod 2^64");
  }
  int done = 0;
  if (int r = streamed_run(G, init_host, seed, max_rounds, (uint8_t*)workspace, ws_bytes,
                           (hipStream_t)stream, color_out_host, k_out, rounds_out, &done))
    return r;
  if (done == 2) return fail(WL_EMAXROUNDS, "no stable colouring after %u rounds", *rounds_out);
  return WL_OK;
}

int wl_verify_workspace_size(const wl_csr* g, uint64_t* bytes_out) {
  g_err[0] = 0;
  if (!g || !bytes_out) return fail(WL_EINVAL, "NULL argument");
  if (g->n >= (1ull << 32)) return fail(WL_EOVERFLOW, "n does not fit 32 bits");
  *bytes_out = ver_layout(g->n, g->nnz, g->weight != nullptr).total;
  return WL_OK;
}

int wl_verify_stable(const wl_csr* g, const uint32_t* color, uint32_t k,
                     void* workspace, uint64_t ws_bytes, void* stream) {
  g_err[0] = 0;
  if (int r = check_graph(g)) return r;
  if (g->n == 0) return WL_OK;
  if (!color) return fail(WL_EINVAL, "color is NULL");
  if (k == 0 || k > g->n) return fail(WL_EINVAL, "k = %u must be in [1, n]", k);
  if (g->nnz > 0 && g->weight == nullptr && g->col_idx == nullptr)
    return fail(WL_EINVAL, "col_idx is NULL");
  const VerLayout L = ver_layout(g->n, g->nnz, g->weight != nullptr);
  if (!workspace) return fail(WL_EINVAL, "workspace is NULL");
  if ((uintptr_t)workspace % kAlign)
    return fail(WL_EINVAL, "workspace must be %llu-byte aligned", (unsigned long long)kAlign);
  if (ws_bytes < L.total)
    return fail(WL_EBUDGET, "workspace has %llu bytes, %llu needed",
                (unsigned long long)ws_bytes, (unsigned long long)L.total);
  hipStream_t s = (hipStream_t)stream;
  if (int r = check_nnz_device(g, s)) return r;
  if (g->weight)
    return verify_run<uint64_t>(g, color, k, (uint8_t*)workspace, L, s);
  return verify_run<uint32_t>(g, color, k, (uint8_t*)workspace, L, s);
}

}  // extern "C"
