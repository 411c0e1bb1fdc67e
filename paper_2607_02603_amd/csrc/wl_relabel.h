// Relabel step of Algorithm 1 (Section 4.1): the new colour of node i is the
// rank of the pair (c_i, z_i) among the distinct pairs in lexicographic order.
//
// The nodes are kept grouped by colour in 'perm' (class c occupies
// perm[cstart[c] .. cstart[c+1])), in increasing colour order.  So the
// lexicographic order of the pairs is: class order, then z inside a class,
// and the relabel is a segmented sort of z inside every class of two or more
// nodes:
//   - classes (and later buckets) of at most kSmallMax nodes are sorted in
//     LDS by one workgroup (a counting sort, or a bitonic network; 8 and 64
//     nodes or fewer: bitonic networks across lanes);
//   - larger ones go through most-significant-digit radix passes over 8-bit
//     digits of z; a bucket whose smallest and largest key agree is finished
//     at once (equal keys need no order), which is the common case in early
//     rounds where a large class has few distinct images.
// Order inside a group of equal pairs is irrelevant, so the passes scatter
// with atomics.  A byte flag marks the first position of every group; an
// inclusive scan of the flags gives the ranks; 'cstart' and 'perm' become the
// grouping of the next round.
#pragma once
#include "wl_block.h"

namespace wl {

// DevState::done of a device-driven round that stopped for the host to finish
// its radix passes, or (kHaltedShift) to build the per-colour shift table of
// a round with more splits than the LDS search takes (k_resume clears both).
constexpr uint32_t kHalted = 3;
constexpr uint32_t kHaltedShift = 4;

// Digit of a radix pass: 8-bit digits from the top of the key (61-bit
// residues of F_p, or 64-bit values of Z/2^64), the last one shorter for F_p.
__device__ __forceinline__ uint32_t digit_of(uint64_t key, int pass, uint32_t ring) {
  const int hi = (ring ? 64 : 61) - kRadixBits * pass;
  const int lo = hi > kRadixBits ? hi - kRadixBits : 0;
  return (uint32_t)((key >> lo) & ((1ull << (hi - lo)) - 1));
}

__global__ void k_round_begin(Ctx ctx) {
  DevState* st = ctx.st;
  if (st->done) return;
  st->n_small = 0;
  st->n_tiny = 0;
  st->n_pico = 0;
  st->n_msort = 0;
  st->big[0] = 0;
  st->big[1] = 0;
  for (int i = 0; i < 4; ++i) st->tickets[i] = 0;
  st->act_entries = 0;
  st->n_split = 0;
  st->n_mid = 0;
  st->n_hlive = 0;
}

__global__ void __launch_bounds__(kBlock) k_fill_u8(Ctx ctx, uint8_t* p,
                                                    uint64_t cnt, uint8_t v) {
  if (ctx.st->done) return;
  for (uint64_t i = blockIdx.x * (uint64_t)kBlock + threadIdx.x; i < cnt;
       i += (uint64_t)gridDim.x * kBlock)
    p[i] = v;
}

__device__ __forceinline__ const uint2* big_list(const Ctx& c, int which) {
  return which ? c.big_list1 : c.big_list0;
}
__device__ __forceinline__ uint2* big_list_w(const Ctx& c, int which) {
  return which ? c.big_list1 : c.big_list0;
}
__device__ __forceinline__ uint32_t* tile_offsets(const Ctx& c, int which) {
  return which ? c.tile_off1 : c.tile_off0;
}
__device__ __forceinline__ uint32_t big_count(const DevState* st, int which) {
  return (uint32_t)(st->big[which] >> 32);
}
__device__ __forceinline__ uint32_t big_tiles(const DevState* st, int which) {
  return (uint32_t)st->big[which];
}

// Appends segment (s, len) to big list 'which' with its first tile: the
// 64-bit add bumps the entry count (high word) by one and the tile count
// (low word) by the segment's tiles, so the returned pair is the segment's
// slot and its first tile, and tile offsets grow with the slot.  The tile
// count stays below 2^32 (at most one tile per kTile nodes plus one per
// segment), so the low word never carries into the high one.
__device__ __forceinline__ void big_append(const Ctx& ctx, int which, uint32_t s,
                                           uint32_t len) {
  const unsigned long long o =
      atomicAdd(&ctx.st->big[which], (1ull << 32) | ((len + kTile - 1) / kTile));
  const uint32_t at = (uint32_t)(o >> 32);
  big_list_w(ctx, which)[at] = make_uint2(s, len);
  tile_offsets(ctx, which)[at] = (uint32_t)o;
}

// One entry per class: flag its first position, queue it if it has >= 2
// members (small classes for the LDS sort, big ones for the radix passes).
__global__ void __launch_bounds__(kBlock) k_segments(Ctx ctx) {
  DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t k = st->k;
  const uint32_t stride = gridDim.x * kBlock;
  for (uint32_t j0 = blockIdx.x * kBlock; j0 < k; j0 += stride) {
    const uint32_t j = j0 + threadIdx.x;
    uint32_t s = 0, len = 0;
    if (j < k) {
      s = ctx.cstart[j];
      const uint32_t e = ctx.cstart[j + 1];
      len = e > s ? e - s : 0;
      if (len) ctx.flags[s] = 1;
    }
    const uint32_t mat = ctx.keys_mat ? kMatBit : 0u;
    // 0 pico, 1 tiny, 2 mid, 3 small, 4 big, 5 none
    const uint32_t kind = len < 2 ? 5u
                          : len <= kPicoMax ? 0u
                          : len <= kTinyMax ? 1u
                          : len <= kMidMax ? 2u
                          : len <= kSmallMax ? 3u : 4u;
    const uint32_t at =
        block_append4(kind, &st->n_pico, &st->n_tiny, &st->n_msort, &st->n_small);
    if (kind == 0) ctx.tiny_list[ctx.max_small - 1 - at] = make_uint2(s, len | mat);
    else if (kind == 1) ctx.tiny_list[at] = make_uint2(s, len | mat);
    else if (kind == 2) ctx.small_list[ctx.max_sm - 1 - at] = make_uint2(s, len | mat);
    else if (kind == 3) ctx.small_list[at] = make_uint2(s, len | mat);
    else if (kind == 4) big_append(ctx, 0, s, len);
  }
}

// Segment index of tile t: last i with off[i] <= t.
__device__ __forceinline__ uint32_t tile_segment(const uint32_t* off,
                                                 uint32_t nb, uint32_t t) {
  uint32_t lo = 0, hi = nb - 1;
  while (lo < hi) {
    uint32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= t)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

struct TileRange {
  uint32_t seg, beg, end, seg_start;
};

__device__ __forceinline__ TileRange tile_range(const Ctx& ctx, int cur,
                                                uint32_t nb, uint32_t t) {
  const uint2* L = big_list(ctx, cur);
  TileRange r;
  const uint32_t* off = tile_offsets(ctx, cur);
  r.seg = tile_segment(off, nb, t);
  const uint2 s = L[r.seg];
  r.seg_start = s.x;
  r.beg = s.x + (t - off[r.seg]) * kTile;
  r.end = min(s.x + s.y, r.beg + kTile);
  return r;
}

// Order in which the workgroups of a radix pass take the tiles: the i-th
// tile taken is (i * (2^31 - 1)) mod nt, a bijection of [0, nt) (2^31 - 1 is
// prime and nt < 2^31).  Workgroups running at one time then hold tiles of
// many segments instead of consecutive tiles of one, so fewer of them
// reserve slots on the same bucket cursors at once.
__device__ __forceinline__ uint32_t tile_order(uint32_t i, uint32_t nt) {
  return (uint32_t)(((uint64_t)i * 2147483647ull) % nt);
}

// First pass only: keys of the big segments in position order.
__global__ void __launch_bounds__(kBlock) k_big_gather(Ctx ctx) {
  DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t nb = big_count(st, 0), nt = big_tiles(st, 0);
  if (nb == 0) return;
  for (uint32_t t = blockIdx.x; t < nt; t += gridDim.x) {
    TileRange r = tile_range(ctx, 0, nb, t);
    for (uint32_t p = r.beg + threadIdx.x; p < r.end; p += kBlock)
      ctx.keys[p] = ctx.z[ctx.perm[p]];
  }
}

// Clears the radix histograms over their whole capacity (max_big segments),
// whatever the state: once per call, before its first radix pass.  From
// then on every k_big_scan clears what it consumed, so each pass finds them
// cleared however many segments it has.
__global__ void __launch_bounds__(kBlock) k_big_clear(Ctx ctx) {
  const uint64_t tot = (uint64_t)ctx.max_big * kRadix;
  for (uint64_t i = blockIdx.x * (uint64_t)kBlock + threadIdx.x; i < tot;
       i += (uint64_t)gridDim.x * kBlock) {
    ctx.bhist[i] = 0;
    ctx.bmin[i] = ~0ull;
    ctx.bmax[i] = 0;
  }
}

// Histogram of the pass digit per (segment, bucket), with min/max key, into
// arrays that k_big_clear and k_big_scan keep cleared.
__global__ void __launch_bounds__(kBlock) k_big_hist(Ctx ctx, int pass) {
  DevState* st = ctx.st;
  if (st->done) return;
  const int cur = pass & 1;
  // the list this pass's k_big_scan fills starts empty (the previous pass
  // consumed it; with nothing left it must not be taken for a later pass)
  if (blockIdx.x == 0 && threadIdx.x == 0) st->big[cur ^ 1] = 0;
  const uint32_t nb = big_count(st, cur), nt = big_tiles(st, cur);
  if (nb == 0) return;
  __shared__ uint32_t cnt[kRadix];
  __shared__ unsigned long long mn[kRadix], mx[kRadix];
  for (uint32_t i = blockIdx.x; i < nt; i += gridDim.x) {
    TileRange r = tile_range(ctx, cur, nb, tile_order(i, nt));
    cnt[threadIdx.x] = 0;
    mn[threadIdx.x] = ~0ull;
    mx[threadIdx.x] = 0;
    __syncthreads();
    // runs of one digit among a thread's keys are counted in registers and
    // added with one set of atomics (classes with few distinct keys give
    // long runs; the LDS atomics of a wave would all hit one bucket).  The
    // thread's keys of the tile are loaded together first.
    uint64_t kv[kTilePerThread];
#pragma unroll
    for (uint32_t q = 0; q < kTilePerThread; ++q) {
      const uint32_t p = r.beg + q * kBlock + threadIdx.x;
      kv[q] = p < r.end ? ctx.keys[p] : 0ull;
    }
    uint32_t rd = 0xFFFFFFFFu, rc = 0;
    unsigned long long rmn = ~0ull, rmx = 0;
#pragma unroll
    for (uint32_t q = 0; q < kTilePerThread; ++q) {
      if (r.beg + q * kBlock + threadIdx.x >= r.end) break;
      const uint64_t key = kv[q];
      const uint32_t d = digit_of(key, pass, ctx.ring);
      if (d != rd) {
        if (rc) {
          atomicAdd(&cnt[rd], rc);
          atomicMin(&mn[rd], rmn);
          atomicMax(&mx[rd], rmx);
        }
        rd = d;
        rc = 0;
        rmn = ~0ull;
        rmx = 0;
      }
      ++rc;
      rmn = key < rmn ? key : rmn;
      rmx = key > rmx ? key : rmx;
    }
    if (rc) {
      atomicAdd(&cnt[rd], rc);
      atomicMin(&mn[rd], rmn);
      atomicMax(&mx[rd], rmx);
    }
    __syncthreads();
    const uint32_t b = threadIdx.x;
    if (cnt[b]) {
      const uint32_t g = r.seg * kRadix + b;
      atomicAdd(&ctx.bhist[g], cnt[b]);
      atomicMin(&ctx.bmin[g], mn[b]);
      atomicMax(&ctx.bmax[g], mx[b]);
    }
    __syncthreads();
  }
}

// One block per big segment: bucket offsets, flags at bucket starts, and the
// follow-up work: finished (one key), LDS sort, or another radix pass.
__global__ void __launch_bounds__(kBlock) k_big_scan(Ctx ctx, int pass) {
  DevState* st = ctx.st;
  if (st->done) return;
  const int cur = pass & 1;
  const uint32_t nb = big_count(st, cur);
  const uint2* L = big_list(ctx, cur);
  __shared__ uint32_t sh[kBlock / kWave];
  for (uint32_t sgi = blockIdx.x; sgi < nb; sgi += gridDim.x) {
    const uint2 s = L[sgi];
    const uint32_t g = sgi * kRadix + threadIdx.x;
    const uint32_t h = ctx.bhist[g];
    const unsigned long long bmn = ctx.bmin[g], bmx = ctx.bmax[g];
    // the histogram is consumed here: leave it cleared for the next pass
    ctx.bhist[g] = 0;
    ctx.bmin[g] = ~0ull;
    ctx.bmax[g] = 0;
    uint32_t tot;
    const uint32_t off = block_excl_scan(h, sh, &tot);
    ctx.bcur[g] = off;
    // every key of the segment equal (one bucket, min == max): its elements
    // are not moved.  Exactly one thread decides (the bucket holding all of
    // them, or bucket 0 when none does).
    const bool all_here = h == s.y;
    const bool none_full = __syncthreads_or(all_here) == 0;
    if (all_here) ctx.bsame[sgi] = bmn == bmx ? 1 : 0;
    else if (none_full && threadIdx.x == 0) ctx.bsame[sgi] = 0;
    const uint32_t pos = s.x + off;
    if (h) ctx.flags[pos] = 1;
    // buckets of two or more distinct keys are sorted further; the list
    // slots of the workgroup's buckets are taken with one atomic per list
    // 0 pico, 1 tiny, 2 mid, 3 small, 4 big, 5 none
    const uint32_t kind = !(h >= 2 && bmn != bmx) ? 5u
                          : h <= kPicoMax ? 0u
                          : h <= kTinyMax ? 1u
                          : h <= kMidMax ? 2u
                          : h <= kSmallMax ? 3u : 4u;
    const uint32_t at =
        block_append4(kind, &st->n_pico, &st->n_tiny, &st->n_msort, &st->n_small);
    if (kind == 0) ctx.tiny_list[ctx.max_small - 1 - at] = make_uint2(pos, h | kMatBit);
    else if (kind == 1) ctx.tiny_list[at] = make_uint2(pos, h | kMatBit);
    else if (kind == 2) ctx.small_list[ctx.max_sm - 1 - at] = make_uint2(pos, h | kMatBit);
    else if (kind == 3) ctx.small_list[at] = make_uint2(pos, h | kMatBit);
    else if (kind == 4) big_append(ctx, cur ^ 1, pos, h);
  }
}

// Scatter every element of the big segments into its bucket (keys_tmp,
// perm_tmp).  A tile's elements are ranked inside their buckets with LDS
// atomics, each bucket's run is reserved with one atomic on its cursor, and
// the elements are staged in LDS in bucket order and written out one per
// lane, consecutive over the lanes, so a wave's stores cover whole runs.
__global__ void __launch_bounds__(kBlock) k_big_scatter(Ctx ctx, int pass) {
  DevState* st = ctx.st;
  if (st->done) return;
  const int cur = pass & 1;
  const uint32_t nb = big_count(st, cur), nt = big_tiles(st, cur);
  if (nb == 0) return;
  __shared__ uint32_t lcnt[kRadix];
  __shared__ uint32_t dbase[kRadix];  // output position of staged slot 0 of the bucket
  __shared__ unsigned long long skey[kTile];
  __shared__ uint32_t sval[kTile];
  __shared__ uint8_t sdig[kTile];
  __shared__ uint32_t sh[kBlock / kWave];
  static_assert(kRadix == kBlock, "one thread per bucket");
  for (uint32_t i = blockIdx.x; i < nt; i += gridDim.x) {
    TileRange r = tile_range(ctx, cur, nb, tile_order(i, nt));
    if (ctx.bsame[r.seg]) continue;  // uniform across the block
    lcnt[threadIdx.x] = 0;
    __syncthreads();
    uint32_t slot[kTilePerThread];
    uint32_t dg[kTilePerThread];
    unsigned long long kv[kTilePerThread];
#pragma unroll
    for (uint32_t q = 0; q < kTilePerThread; ++q) {
      const uint32_t p = r.beg + q * kBlock + threadIdx.x;
      if (p < r.end) {
        kv[q] = ctx.keys[p];
        dg[q] = digit_of(kv[q], pass, ctx.ring);
        slot[q] = atomicAdd(&lcnt[dg[q]], 1u);
      }
    }
    __syncthreads();
    const uint32_t b = threadIdx.x;
    const uint32_t h = lcnt[b];
    uint32_t tot;
    const uint32_t lofs = block_excl_scan(h, sh, &tot);
    const uint32_t gb = h ? atomicAdd(&ctx.bcur[r.seg * kRadix + b], h) : 0u;
    // u32 arithmetic: the difference may wrap, the sum with a slot does not
    dbase[b] = r.seg_start + gb - lofs;
    lcnt[b] = lofs;
    __syncthreads();
#pragma unroll
    for (uint32_t q = 0; q < kTilePerThread; ++q) {
      const uint32_t p = r.beg + q * kBlock + threadIdx.x;
      if (p < r.end) {
        const uint32_t at = lcnt[dg[q]] + slot[q];
        skey[at] = kv[q];
        sval[at] = ctx.perm[p];
        sdig[at] = (uint8_t)dg[q];
      }
    }
    __syncthreads();
    const uint32_t cnt = r.end - r.beg;
    for (uint32_t t = threadIdx.x; t < cnt; t += kBlock) {
      const uint32_t dst = dbase[sdig[t]] + t;
      ctx.keys_tmp[dst] = skey[t];
      ctx.perm_tmp[dst] = sval[t];
    }
    __syncthreads();
  }
}

__global__ void __launch_bounds__(kBlock) k_big_copyback(Ctx ctx, int pass) {
  DevState* st = ctx.st;
  if (st->done) return;
  const int cur = pass & 1;
  const uint32_t nb = big_count(st, cur), nt = big_tiles(st, cur);
  if (nb == 0) return;
  for (uint32_t t = blockIdx.x; t < nt; t += gridDim.x) {
    TileRange r = tile_range(ctx, cur, nb, t);
    if (ctx.bsame[r.seg]) continue;
    // all loads of the thread's share of the tile before its stores
    uint64_t kv[kTilePerThread];
    uint32_t pv[kTilePerThread];
#pragma unroll
    for (uint32_t q = 0; q < kTilePerThread; ++q) {
      const uint32_t p = r.beg + q * kBlock + threadIdx.x;
      if (p < r.end) {
        kv[q] = ctx.keys_tmp[p];
        pv[q] = ctx.perm_tmp[p];
      }
    }
#pragma unroll
    for (uint32_t q = 0; q < kTilePerThread; ++q) {
      const uint32_t p = r.beg + q * kBlock + threadIdx.x;
      if (p < r.end) {
        ctx.keys[p] = kv[q];
        ctx.perm[p] = pv[q];
      }
    }
  }
}

// Order of the sorting networks below.  Padding slots carry the largest key
// ~0 and node 0xFFFFFFFF (no node has that id).  In F_p no key reaches ~0,
// so keys alone decide (TIE = false).  In Z/2^64 a key may equal ~0: then
// (key, node) pairs are compared (TIE = true), which keeps every padding slot
// behind every node.
template <bool TIE>
__device__ __forceinline__ bool key_less(unsigned long long a, uint32_t va,
                                         unsigned long long b, uint32_t vb) {
  return a < b || (TIE && a == b && va < vb);
}

constexpr uint32_t kCsBits = 10, kCsBuckets = 1u << kCsBits, kCsFix = 32;
static_assert(kSmallMax <= 65536 && kCsBuckets % kBlock == 0, "counting sort of small segments");

// LDS of one small-segment sort (one workgroup).
struct SmallLds {
  unsigned long long skey[kSmallMax];
  uint32_t sval[kSmallMax];
  uint32_t cnt[kCsBuckets + 1];
  uint16_t inv[kSmallMax];
  uint8_t mixed[kCsBuckets];
  unsigned long long xo;
  uint32_t csh[kBlock / kWave];
  int differ, unsorted, fallback;
};

// One workgroup per small segment, keys in LDS: a counting sort by the ten
// bits at and below the highest bit in which the keys differ, whose mixed
// buckets of at most ctx.cs_fix (default kCsFix) keys are sorted by insertion;
// a larger mixed bucket (rare for hashed images) falls back to a bitonic sort
// of (z, node).
// Then flags where z changes.
// 'extra' mid segments (from the back of the list) are sorted here too.
template <bool TIE>
__device__ __forceinline__ void small_sort_body(const Ctx& ctx, SmallLds& L, uint32_t bid,
                                                uint32_t nblk, uint32_t extra) {
  DevState* st = ctx.st;
  const uint32_t ns = st->n_small;
  unsigned long long* const skey = L.skey;
  uint32_t* const sval = L.sval;
  uint32_t* const cnt = L.cnt;
  uint16_t* const inv = L.inv;
  uint8_t* const mixed = L.mixed;
  uint32_t* const csh = L.csh;
  unsigned long long& xo = L.xo;
  int& differ = L.differ;
  int& unsorted = L.unsorted;
  int& fallback = L.fallback;
  for (uint32_t si = bid; si < ns + extra; si += nblk) {
    const uint2 sg = si < ns ? ctx.small_list[si] : ctx.small_list[ctx.max_sm - 1 - (si - ns)];
    const uint32_t s = sg.x, len = sg.y & ~kMatBit;
    const bool mat = (sg.y & kMatBit) != 0;
    uint32_t P = 2;
    while (P < len) P <<= 1;
    // the segment into LDS; the flags and the bucket counts of the counting
    // sort below are cleared on the way (nothing reads them before the
    // barrier)
    if (threadIdx.x == 0) {
      differ = 0;
      unsorted = 0;
      xo = 0;
      fallback = 0;
    }
    for (uint32_t b = threadIdx.x; b < kCsBuckets; b += kBlock) {
      cnt[b] = 0;
      mixed[b] = 0;
    }
    for (uint32_t t = threadIdx.x; t < P; t += kBlock) {
      if (t < len) {
        const uint32_t v = ctx.perm[s + t];
        sval[t] = v;
        skey[t] = mat ? ctx.keys[s + t] : ctx.z[v];
      } else {
        sval[t] = 0xFFFFFFFFu;
        skey[t] = ~0ull;
      }
    }
    __syncthreads();
    // all images equal: nothing splits, nothing to reorder; already in
    // order (the rows of a quotient): only the flags.  The same pass ORs the
    // differences to the first key (the highest differing bit, below).
    {
      unsigned long long x = 0;
      bool uns = false;
      for (uint32_t t = threadIdx.x; t < len; t += kBlock) {
        x |= skey[t] ^ skey[0];
        uns = uns || (t + 1 < len && key_less<TIE>(skey[t + 1], sval[t + 1], skey[t], sval[t]));
      }
      if (x) {
        differ = 1;
        atomicOr(&xo, x);
      }
      if (uns) unsorted = 1;
    }
    __syncthreads();
    if (!differ) {
      // every thread has read the flag before the next segment clears it
      __syncthreads();
      continue;
    }
    if (!unsorted) {
      for (uint32_t t = threadIdx.x + 1; t < len; t += kBlock)
        if (skey[t] != skey[t - 1]) ctx.flags[s + t] = 1;
      __syncthreads();
      continue;
    }
    // Counting sort by the kCsBits bits at and below the highest bit in which
    // the keys differ (above it they all agree), into inv (position ->
    // element); then a bucket whose keys are not all equal is sorted by
    // insertion when it holds at most ctx.cs_fix keys, and a larger one sends the
    // segment to the sorting network below.
    const int top = 63 - __clzll((long long)xo);  // xo != 0: the keys differ
    const int sh = top >= (int)kCsBits - 1 ? top - ((int)kCsBits - 1) : 0;
    uint32_t rk[kSmallMax / kBlock];
#pragma unroll
    for (uint32_t j = 0; j < kSmallMax / kBlock; ++j) {
      const uint32_t t = threadIdx.x + j * kBlock;
      if (t < len) rk[j] = atomicAdd(&cnt[(skey[t] >> sh) & (kCsBuckets - 1)], 1u);
    }
    __syncthreads();
    {
      // exclusive scan of the counts, kCsBuckets / kBlock per thread; cnt[kCsBuckets] = len
      constexpr uint32_t kPer = kCsBuckets / kBlock;
      uint32_t c[kPer], sum = 0;
#pragma unroll
      for (uint32_t u = 0; u < kPer; ++u) {
        c[u] = cnt[threadIdx.x * kPer + u];
        sum += c[u];
      }
      uint32_t tot;
      uint32_t run = block_excl_scan(sum, csh, &tot);
#pragma unroll
      for (uint32_t u = 0; u < kPer; ++u) {
        cnt[threadIdx.x * kPer + u] = run;
        run += c[u];
      }
      if (threadIdx.x == 0) cnt[kCsBuckets] = len;
    }
    __syncthreads();
#pragma unroll
    for (uint32_t j = 0; j < kSmallMax / kBlock; ++j) {
      const uint32_t t = threadIdx.x + j * kBlock;
      if (t < len) inv[cnt[(skey[t] >> sh) & (kCsBuckets - 1)] + rk[j]] = (uint16_t)t;
    }
    __syncthreads();
    for (uint32_t p = threadIdx.x + 1; p < len; p += kBlock) {
      const unsigned long long k = skey[inv[p]];
      const uint32_t d = (uint32_t)(k >> sh) & (kCsBuckets - 1);
      if (p > cnt[d] && k != skey[inv[p - 1]]) mixed[d] = 1;
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < kCsBuckets; b += kBlock) {
      if (!mixed[b]) continue;
      const uint32_t o = cnt[b], c = cnt[b + 1] - o;
      if (c > ctx.cs_fix) {
        fallback = 1;
        continue;
      }
      for (uint32_t i = o + 1; i < o + c; ++i) {
        const uint16_t e = inv[i];
        const unsigned long long k = skey[e];
        uint32_t j = i;
        while (j > o && skey[inv[j - 1]] > k) {
          inv[j] = inv[j - 1];
          --j;
        }
        inv[j] = e;
      }
    }
    __syncthreads();
    if (!fallback) {
      for (uint32_t p = threadIdx.x; p < len; p += kBlock) {
        const uint32_t t = inv[p];
        ctx.perm[s + p] = sval[t];
        if (mat) ctx.keys[s + p] = skey[t];
        if (p > 0 && skey[t] != skey[inv[p - 1]]) ctx.flags[s + p] = 1;
      }
      __syncthreads();
      continue;
    }
    for (uint32_t kk = 2; kk <= P; kk <<= 1) {
      for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
        for (uint32_t i = threadIdx.x; i < P; i += kBlock) {
          const uint32_t l = i ^ j;
          if (l > i) {
            const bool asc = (i & kk) == 0;
            const unsigned long long a = skey[i], b = skey[l];
            if (key_less<TIE>(b, sval[l], a, sval[i]) == asc) {
              skey[i] = b;
              skey[l] = a;
              const uint32_t tv = sval[i];
              sval[i] = sval[l];
              sval[l] = tv;
            }
          }
        }
        __syncthreads();
      }
    }
    for (uint32_t t = threadIdx.x; t < len; t += kBlock) {
      ctx.perm[s + t] = sval[t];
      if (mat) ctx.keys[s + t] = skey[t];  // sorted keys stay with their payload
      if (t > 0 && skey[t] != skey[t - 1]) ctx.flags[s + t] = 1;
    }
    __syncthreads();
  }
}

// One wave per tiny segment (<= 64 nodes): bitonic sort of (z, node) across
// the lanes with shuffles, flags where z changes.  Skipped when all images of
// the segment are equal.
// check_passes >= 0: first halt the device (done = kHalted) if big segments
// are left after that many radix passes; the workgroups of the launch that
// still run (of all three sorts) sort their segments, which the host-driven
// completion sorts again (the keys stay in order; only members with equal
// keys may change places, and their order is irrelevant).
template <bool TIE>
__device__ __forceinline__ void tiny_sort_body(const Ctx& ctx, int check_passes, uint32_t bid,
                                               uint32_t nblk) {
  DevState* st = ctx.st;
  if (check_passes >= 0 && bid == 0 && threadIdx.x == 0 && big_count(st, check_passes & 1) > 0)
    st->done = kHalted;
  const uint32_t nt = st->n_tiny;
  const uint32_t lane = lane_id();
  const uint32_t nwaves = nblk * (kBlock / kWave);
  for (uint32_t si = bid * (kBlock / kWave) + threadIdx.x / kWave; si < nt;
       si += nwaves) {
    const uint2 sg = ctx.tiny_list[si];
    const uint32_t s = sg.x, len = sg.y & ~kMatBit;
    const bool mat = (sg.y & kMatBit) != 0;
    unsigned long long key = ~0ull;
    uint32_t v = 0xFFFFFFFFu;
    if (lane < len) {
      v = ctx.perm[s + lane];
      key = mat ? ctx.keys[s + lane] : ctx.z[v];
    }
    const unsigned long long first = __shfl(key, 0, kWave);
    if (__ballot(lane < len && key != first) == 0) continue;
#pragma unroll
    for (uint32_t kk = 2; kk <= (uint32_t)kWave; kk <<= 1) {
#pragma unroll
      for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
        const unsigned long long pk = __shfl_xor(key, (int)j, kWave);
        const uint32_t pv = __shfl_xor(v, (int)j, kWave);
        const bool up = (lane & kk) == 0;
        const bool lower = (lane & j) == 0;
        const bool take =
            (lower == up) ? key_less<TIE>(pk, pv, key, v) : key_less<TIE>(key, v, pk, pv);
        if (take) {
          key = pk;
          v = pv;
        }
      }
    }
    const unsigned long long prev = __shfl_up(key, 1, kWave);
    if (lane < len) {
      ctx.perm[s + lane] = v;
      if (mat) ctx.keys[s + lane] = key;  // sorted keys stay with their payload
      if (lane > 0 && key != prev) ctx.flags[s + lane] = 1;
    }
  }
}

// Segments of at most kPicoMax nodes, listed from the back of the tiny
// list: eight per wave, eight lanes each, with the tiny sort's bitonic
// network cut to eight elements.  Skipped when all keys of a segment agree.
template <bool TIE>
__device__ __forceinline__ void pico_sort_body(const Ctx& ctx, uint32_t bid, uint32_t nblk) {
  DevState* st = ctx.st;
  const uint32_t np = st->n_pico;
  const uint32_t lane = lane_id(), sub = lane & 7u, g0 = lane & ~7u;
  const uint32_t nwaves = nblk * (kBlock / kWave);
  // loop bounds are the same for the whole wave (the shuffles need every lane)
  for (uint32_t base = (bid * (kBlock / kWave) + threadIdx.x / kWave) * 8; base < np;
       base += nwaves * 8) {
    const uint32_t si = base + (lane >> 3);
    uint32_t s = 0, len = 0;
    bool mat = false;
    if (si < np) {
      const uint2 sg = ctx.tiny_list[ctx.max_small - 1 - si];
      s = sg.x;
      len = sg.y & ~kMatBit;
      mat = (sg.y & kMatBit) != 0;
    }
    unsigned long long key = ~0ull;
    uint32_t v = 0xFFFFFFFFu;
    if (sub < len) {
      v = ctx.perm[s + sub];
      key = mat ? ctx.keys[s + sub] : ctx.z[v];
    }
    const unsigned long long first = __shfl(key, (int)g0, kWave);
    const unsigned long long dm = __ballot(sub < len && key != first);
    const bool differ = ((dm >> g0) & 0xFFull) != 0;
#pragma unroll
    for (uint32_t kk = 2; kk <= 8; kk <<= 1) {
#pragma unroll
      for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
        const unsigned long long pk = __shfl_xor(key, (int)j, kWave);
        const uint32_t pv = __shfl_xor(v, (int)j, kWave);
        const bool up = (sub & kk) == 0;
        const bool lower = (sub & j) == 0;
        const bool take =
            (lower == up) ? key_less<TIE>(pk, pv, key, v) : key_less<TIE>(key, v, pk, pv);
        if (take) {
          key = pk;
          v = pv;
        }
      }
    }
    const unsigned long long prev = __shfl_up(key, 1, kWave);
    if (differ && sub < len) {
      ctx.perm[s + sub] = v;
      if (mat) ctx.keys[s + sub] = key;
      if (sub > 0 && key != prev) ctx.flags[s + sub] = 1;
    }
  }
}

// Segments of kTinyMax + 1 .. kMidMax keys, one wave each (four per
// workgroup, no workgroup barrier): a counting sort in LDS on the kMidBits
// bits at and below the highest bit in which the keys differ, lane l owning
// buckets kMidPer * l ..; a bucket whose keys differ is sorted by its lane by
// insertion when it holds at most ctx.cs_fix keys (as in the small sort), and
// a larger one sends the segment to a bitonic network in LDS.  A wave's LDS accesses are ordered by
// the wave itself (the LDS executes a wave's instructions in order); the
// fences only keep the compiler from moving them across a step.
constexpr uint32_t kMidBits = 9, kMidBuckets = 1u << kMidBits;
constexpr uint32_t kMidWaves = 1024;  // fewer mid segments go to the workgroup sort
constexpr uint32_t kMidPer = kMidMax / kWave;  // keys, and buckets, per lane
static_assert(kMidBuckets == kMidMax, "one bucket per key slot: lane l owns the same range of both");

struct MidLds {  // one wave
  unsigned long long skey[kMidMax];
  uint32_t sval[kMidMax];
  uint32_t cnt[kMidBuckets + 1];
  uint16_t inv[kMidMax];
};

__device__ __forceinline__ void wave_lds_step() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <bool TIE>
__device__ __forceinline__ void mid_sort_body(const Ctx& ctx, MidLds* lds, uint32_t bid,
                                              uint32_t nblk) {
  const DevState* st = ctx.st;
  const uint32_t nm = st->n_msort;
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  MidLds& L = lds[w];
  const uint32_t nwaves = nblk * (kBlock / kWave);
  for (uint32_t si = bid * (kBlock / kWave) + w; si < nm; si += nwaves) {
    const uint2 sg = ctx.small_list[ctx.max_sm - 1 - si];
    const uint32_t s = sg.x, len = sg.y & ~kMatBit;
    const bool mat = (sg.y & kMatBit) != 0;
    // entry t = lane + kWave * u of the segment in registers
    unsigned long long kr[kMidPer];
    uint32_t vr[kMidPer];
#pragma unroll
    for (uint32_t u = 0; u < kMidPer; ++u) {
      const uint32_t t = lane + kWave * u;
      kr[u] = ~0ull;
      vr[u] = 0xFFFFFFFFu;
      if (t < len) {
        vr[u] = ctx.perm[s + t];
        kr[u] = mat ? ctx.keys[s + t] : ctx.z[vr[u]];
      }
    }
    // the bits in which the keys differ from the first (len > kTinyMax: lane 0 holds it)
    const unsigned long long first = read_lane64(kr[0], 0);
    unsigned long long x = 0;
#pragma unroll
    for (uint32_t u = 0; u < kMidPer; ++u)
      if (lane + kWave * u < len) x |= kr[u] ^ first;
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) x |= __shfl_xor(x, off, kWave);
    if (x == 0) continue;  // all equal: nothing to reorder, no flag inside
    const int top = 63 - __clzll((long long)x);
    const int sh = top >= (int)kMidBits - 1 ? top - ((int)kMidBits - 1) : 0;
    // (every lane is past the previous segment's last LDS access: the loop
    // bounds are the same for the whole wave)
#pragma unroll
    for (uint32_t u = 0; u < kMidPer; ++u) {
      const uint32_t t = lane + kWave * u;
      L.cnt[lane * kMidPer + u] = 0;
      if (t < len) {
        L.skey[t] = kr[u];
        L.sval[t] = vr[u];
      }
    }
    wave_lds_step();
    uint32_t rk[kMidPer];
#pragma unroll
    for (uint32_t u = 0; u < kMidPer; ++u)
      if (lane + kWave * u < len)
        rk[u] = atomicAdd(&L.cnt[(kr[u] >> sh) & (kMidBuckets - 1)], 1u);
    wave_lds_step();
    {
      // exclusive scan of the counts; cnt[kMidBuckets] = len
      uint32_t c[kMidPer], sum = 0;
#pragma unroll
      for (uint32_t u = 0; u < kMidPer; ++u) {
        c[u] = L.cnt[lane * kMidPer + u];
        sum += c[u];
      }
      uint32_t run = wave_incl_scan(sum) - sum;
#pragma unroll
      for (uint32_t u = 0; u < kMidPer; ++u) {
        L.cnt[lane * kMidPer + u] = run;
        run += c[u];
      }
      if (lane == 0) L.cnt[kMidBuckets] = len;
    }
    wave_lds_step();
#pragma unroll
    for (uint32_t u = 0; u < kMidPer; ++u) {
      const uint32_t t = lane + kWave * u;
      if (t < len) L.inv[L.cnt[(kr[u] >> sh) & (kMidBuckets - 1)] + rk[u]] = (uint16_t)t;
    }
    wave_lds_step();
    // each lane fixes its own buckets
    bool too_big = false;
#pragma unroll
    for (uint32_t u = 0; u < kMidPer; ++u) {
      const uint32_t b = lane * kMidPer + u;
      const uint32_t o = L.cnt[b], c = L.cnt[b + 1] - o;
      if (c < 2) continue;
      if (c > ctx.cs_fix) {
        for (uint32_t i = o + 1; i < o + c; ++i)
          if (L.skey[L.inv[i]] != L.skey[L.inv[o]]) too_big = true;
        continue;
      }
      for (uint32_t i = o + 1; i < o + c; ++i) {
        const uint16_t e = L.inv[i];
        const unsigned long long k = L.skey[e];
        uint32_t j = i;
        while (j > o && L.skey[L.inv[j - 1]] > k) {
          L.inv[j] = L.inv[j - 1];
          --j;
        }
        L.inv[j] = e;
      }
    }
    wave_lds_step();
    if (__ballot(too_big) == 0) {
#pragma unroll
      for (uint32_t u = 0; u < kMidPer; ++u) {
        const uint32_t p = lane + kWave * u;
        if (p < len) {
          const uint32_t e = L.inv[p];
          ctx.perm[s + p] = L.sval[e];
          if (mat) ctx.keys[s + p] = L.skey[e];
          if (p > 0 && L.skey[e] != L.skey[L.inv[p - 1]]) ctx.flags[s + p] = 1;
        }
      }
      wave_lds_step();
      continue;
    }
    // a bucket of more than cs_fix keys that differ: bitonic network over
    // the segment in LDS, padded with the largest key (node 0xFFFFFFFF)
    uint32_t P = 2;
    while (P < len) P <<= 1;
    for (uint32_t t = len + lane; t < P; t += kWave) {
      L.skey[t] = ~0ull;
      L.sval[t] = 0xFFFFFFFFu;
    }
    wave_lds_step();
    for (uint32_t kk = 2; kk <= P; kk <<= 1)
      for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
        for (uint32_t i = lane; i < P; i += kWave) {
          const uint32_t l = i ^ j;
          if (l > i) {
            const bool asc = (i & kk) == 0;
            const unsigned long long a = L.skey[i], b = L.skey[l];
            const uint32_t va = L.sval[i], vb = L.sval[l];
            if (key_less<TIE>(b, vb, a, va) == asc) {
              L.skey[i] = b;
              L.skey[l] = a;
              L.sval[i] = vb;
              L.sval[l] = va;
            }
          }
        }
        wave_lds_step();
      }
    for (uint32_t t = lane; t < len; t += kWave) {
      ctx.perm[s + t] = L.sval[t];
      if (mat) ctx.keys[s + t] = L.skey[t];
      if (t > 0 && L.skey[t] != L.skey[t - 1]) ctx.flags[s + t] = 1;
    }
    wave_lds_step();
  }
}

// The sorts in one launch: workgroups [0, gt) take the tiny segments,
// [gt, gt + gp) the pico ones and the rest the mid ones and then the small
// ones (each kind in a grid-stride loop over its workgroups).  The mid
// segments take one wave each when there are at least kMidWaves of them
// (throughput); fewer are sorted like the small ones, by whole workgroups,
// which finish one segment sooner.  The mid and small sorts share the
// workgroup's LDS.
template <bool TIE>
__global__ void __launch_bounds__(kBlock) k_sorts(Ctx ctx, int check_passes, uint32_t gt,
                                                  uint32_t gp) {
  if (ctx.st->done) return;
  __shared__ union {
    SmallLds small;
    MidLds mid[kBlock / kWave];
  } lds;
  const uint32_t b = blockIdx.x;
  if (b < gt) {
    tiny_sort_body<TIE>(ctx, check_passes, b, gt);
  } else if (b < gt + gp) {
    pico_sort_body<TIE>(ctx, b - gt, gp);
  } else {
    const uint32_t bid = b - gt - gp, nblk = gridDim.x - gt - gp;
    const uint32_t nm = ctx.st->n_msort;
    const bool by_wave = nm >= kMidWaves;
    if (by_wave) {
      mid_sort_body<TIE>(ctx, lds.mid, bid, nblk);
      __syncthreads();  // every wave is done with the mid LDS
    }
    small_sort_body<TIE>(ctx, lds.small, bid, nblk, by_wave ? 0u : nm);
  }
}

// ---------------------------------------------------------------------------
// Device-wide inclusive scan of the byte flags -> ranks (ids = scan - 1).
// ---------------------------------------------------------------------------

__device__ __forceinline__ void scan_range(uint32_t n, uint32_t b, uint32_t nblk,
                                           uint32_t* lo, uint32_t* hi) {
  const uint32_t per = ((n + nblk - 1) / nblk + kBlock - 1) / kBlock * kBlock;
  *lo = min(n, b * per);
  *hi = min(n, *lo + per);
}

__global__ void __launch_bounds__(kBlock) k_scan_part(Ctx ctx) {
  if (ctx.st->done) return;
  uint32_t lo, hi;
  scan_range(ctx.n, blockIdx.x, gridDim.x, &lo, &hi);
  uint32_t s = 0;
  for (uint32_t p = lo + threadIdx.x; p < hi; p += kBlock) s += ctx.flags[p];
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t tot;
  block_excl_scan(s, sh, &tot);
  if (threadIdx.x == 0) ctx.scan_part[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(kBlock) k_scan_top(Ctx ctx, uint32_t nblk) {
  if (ctx.st->done) return;
  __shared__ uint32_t sh[kBlock / kWave];
  const uint32_t carry = block_scan_small(ctx.scan_part, nblk, sh);
  if (threadIdx.x == 0) ctx.st->k_new = carry;
}

__global__ void __launch_bounds__(kBlock) k_scan_final(Ctx ctx) {
  if (ctx.st->done) return;
  uint32_t lo, hi;
  scan_range(ctx.n, blockIdx.x, gridDim.x, &lo, &hi);
  uint32_t run = ctx.scan_part[blockIdx.x];
  __shared__ uint32_t sh[kBlock / kWave];
  for (uint32_t base = lo; base < hi; base += kBlock) {
    const uint32_t p = base + threadIdx.x;
    const uint32_t f = p < hi ? ctx.flags[p] : 0;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(f, sh, &tot);
    if (p < hi) ctx.ids[p] = run + ex + f - 1;
    run += tot;
  }
}

// New class starts, then colours and activity per node.
// When the colours in use are exactly [0, k) and no class split
// (k_new == k), the ranks equal the old colours: colours, grouping and
// activity are already right and both kernels return.
__global__ void __launch_bounds__(kBlock) k_cstart(Ctx ctx) {
  if (ctx.st->done) return;
  if (ctx.st->dense && ctx.st->k_new == ctx.st->k) return;
  for (uint32_t p = blockIdx.x * kBlock + threadIdx.x; p < ctx.n;
       p += gridDim.x * kBlock)
    if (ctx.flags[p]) ctx.cstart[ctx.ids[p]] = p;
  if (blockIdx.x == 0 && threadIdx.x == 0) ctx.cstart[ctx.st->k_new] = ctx.n;
}

__global__ void __launch_bounds__(kBlock) k_scatter_colors(Ctx ctx) {
  if (ctx.st->done) return;
  if (ctx.st->dense && ctx.st->k_new == ctx.st->k) return;
  for (uint32_t p = blockIdx.x * kBlock + threadIdx.x; p < ctx.n;
       p += gridDim.x * kBlock) {
    const uint32_t v = ctx.perm[p], id = ctx.ids[p];
    ctx.c[v] = id;
    ctx.act[v] = (ctx.cstart[id + 1] - ctx.cstart[id]) >= 2 ? 1 : 0;
  }
}

// Clears the halt of a device-driven round before the host finishes it.
__global__ void k_resume(Ctx ctx) {
  if (ctx.st->done == kHalted || ctx.st->done == kHaltedShift) ctx.st->done = 0;
}

__global__ void k_round_end(Ctx ctx, int count_round) {
  DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t kn = st->k_new;
  if (count_round) {
    st->round += 1;
    if (kn == st->k)
      st->done = 1;
    else if (st->round >= st->max_rounds)
      st->done = 2;
  }
  st->k = kn;
}

}  // namespace wl
