// Relabel step of Algorithm 1 (Section 4.1) restricted to the classes that
// can still split.
//
// New colour of node i = rank of (c_i, z_i) among the distinct pairs in
// lexicographic order.  Colours are dense ranks, so a class b that splits
// into s sub-classes (sorted by z) receives the ids
//     b + shift(b), ..., b + shift(b) + s - 1,
// where shift(b) counts the extra sub-classes created by the classes before
// b, and a class that does not split keeps b + shift(b).  A class can only
// split when it has two or more members and one of them has a non-empty row
// (an empty row has z = 0 in every round), so only such "live" classes are
// sorted; everything else just moves by shift.
//
// State kept between rounds (device):
//   L      live classes in colour order: old colour lcold[j], members at
//          lperm[loff[j] .. loff[j] + llen[j]); qcls[q] = class of position q.
//          The sort permutes lperm with the keys.  A class that does not
//          split is not moved (the sorts leave classes of equal keys alone),
//          so rs/rl stay valid by position for it; the members of classes
//          that split take them from the row pointers.
//   rs, rl first entry and length of the row of every position's node (an
//          empty row has key 0; the image is computed only for the others).
//   act    rows longer than kHeavyChunk use the static heavy chunks, which
//          check act; every round sets it for the heavy rows of live classes.
// One round after the image:
//   load      keys[q] = z of lperm[q] (0 for an empty row)
//   sort      segmented sort of the keys inside every live class (the MSD
//             radix / LDS / wave sorts of wl_relabel.h, keys materialised)
//   scan      flags at sub-class starts (class start, or key change); their
//             inclusive scan R gives the sub-class index g = R - 1 and the
//             new colour lcold[j] + g - j; sub-class extents and whether a
//             sub-class holds a non-empty row
//   shift     classes that split (old colour, extra sub-classes) -> shift(b)
//             for every colour, applied to every node
//   emit      members of live classes get their exact new colour; live
//             sub-classes (>= 2 members, a non-empty row) form the next L.
// Every kernel reads its counts from the device state, so a round can be
// queued without reading anything back.
#pragma once
#include "wl_relabel.h"
#include "wl_spmv.h"

namespace wl {

constexpr uint32_t kShiftLds = 4096;  // splits searched in LDS; more use a table

// ---------------------------------------------------------------------------
// Generic exclusive scan of one or two u32 arrays in place, length read from
// device memory, totals written to device memory.  Two launches of the same
// grid (at most kScanBlocks blocks): part (block sums), final (each block
// sums the block sums below its own, then scans its range).
// ---------------------------------------------------------------------------

// Block b's range [lo, hi) of a scan over len items: a multiple of
// kScanStep items (but the last), so every step of kScanStep items starts
// at a multiple of kScanItems.
constexpr uint32_t kScanItems = 4;                  // consecutive items per thread and step
constexpr uint32_t kScanStep = kScanItems * kBlock;
__device__ __forceinline__ void xscan_range(uint32_t len, uint32_t b, uint32_t nblk,
                                            uint32_t* lo, uint32_t* hi) {
  const uint32_t per = ((len + nblk - 1) / nblk + kScanStep - 1) / kScanStep * kScanStep;
  *lo = (uint32_t)min((uint64_t)len, (uint64_t)b * per);
  *hi = (uint32_t)min((uint64_t)len, (uint64_t)*lo + per);
}

// v[u] = p[i + u] for the u with i + u < n (0 beyond); a whole group is one
// 16-byte load when p + i is 16-byte aligned (i is a multiple of 4 here, so
// that is a property of p alone).
__device__ __forceinline__ void load4(const uint32_t* p, uint32_t i, uint32_t n, uint32_t v[4]) {
  if (i + 3 < n && ((uintptr_t)(p + i) & 15) == 0) {
    const uint4 w = *(const uint4*)(p + i);
    v[0] = w.x;
    v[1] = w.y;
    v[2] = w.z;
    v[3] = w.w;
  } else {
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) v[u] = i + u < n ? p[i + u] : 0u;
  }
}
__device__ __forceinline__ void load4(const uint64_t* p, uint32_t i, uint32_t n, uint64_t v[4]) {
  if (i + 3 < n && ((uintptr_t)(p + i) & 15) == 0) {
    const ulonglong2 w0 = *(const ulonglong2*)(p + i);
    const ulonglong2 w1 = *(const ulonglong2*)(p + i + 2);
    v[0] = w0.x;
    v[1] = w0.y;
    v[2] = w1.x;
    v[3] = w1.y;
  } else {
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) v[u] = i + u < n ? p[i + u] : 0ull;
  }
}

// 'run_if' (device, may be NULL): the scan runs only when *run_if != 0.
__global__ void __launch_bounds__(kBlock) k_xscan_part(const DevState* st, const uint32_t* run_if,
                                                       const uint32_t* lenp, const uint32_t* a,
                                                       const uint32_t* b, uint32_t* part) {
  if (st->done || (run_if && !*run_if)) return;
  uint32_t lo, hi;
  xscan_range(*lenp, blockIdx.x, gridDim.x, &lo, &hi);
  uint32_t sa = 0, sb = 0;
  for (uint32_t i = lo + kScanItems * threadIdx.x; i < hi; i += kScanStep) {
    uint32_t v[4];
    load4(a, i, hi, v);
    sa += v[0] + v[1] + v[2] + v[3];
    if (b) {
      load4(b, i, hi, v);
      sb += v[0] + v[1] + v[2] + v[3];
    }
  }
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t ta, tb = 0;
  block_excl_scan(sa, sh, &ta);
  if (b) block_excl_scan(sb, sh, &tb);
  if (threadIdx.x == 0) {
    part[blockIdx.x] = ta;
    part[gridDim.x + blockIdx.x] = tb;
  }
}

// Totals to *tot_a / *tot_b (either may be NULL) by block 0.
__global__ void __launch_bounds__(kBlock) k_xscan_final(const DevState* st, const uint32_t* run_if,
                                                        const uint32_t* lenp, uint32_t* a,
                                                        uint32_t* b, const uint32_t* part,
                                                        uint32_t* tot_a, uint32_t* tot_b) {
  static_assert(kScanBlocks <= 4 * kBlock, "block sums summed by one block");
  if (st->done || (run_if && !*run_if)) return;
  uint32_t lo, hi;
  xscan_range(*lenp, blockIdx.x, gridDim.x, &lo, &hi);
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t sa, sb = 0;
  uint32_t ra = block_part_prefix(part, gridDim.x, blockIdx.x, sh, &sa);
  uint32_t rb = b ? block_part_prefix(part + gridDim.x, gridDim.x, blockIdx.x, sh, &sb) : 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (tot_a) *tot_a = sa;
    if (tot_b) *tot_b = sb;
  }
  for (uint32_t base = lo; base < hi; base += kScanStep) {
    const uint32_t i = base + kScanItems * threadIdx.x;
    uint32_t va[4], vb[4] = {0, 0, 0, 0};
    load4(a, i, hi, va);
    if (b) load4(b, i, hi, vb);
    uint32_t ta, tb = 0;
    uint32_t xa = ra + block_excl_scan(va[0] + va[1] + va[2] + va[3], sh, &ta);
    uint32_t xb = b ? rb + block_excl_scan(vb[0] + vb[1] + vb[2] + vb[3], sh, &tb) : 0u;
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u)
      if (i + u < hi) {
        a[i + u] = xa;
        xa += va[u];
        if (b) {
          b[i + u] = xb;
          xb += vb[u];
        }
      }
    ra += ta;
    rb += tb;
  }
}

// ---------------------------------------------------------------------------
// Set-up of the live classes from a grouping (perm, cstart, ids = colour of
// every position), once per call after the canonical start.
// ---------------------------------------------------------------------------

template <typename RP>
__device__ __forceinline__ bool row_nonempty(const Ctx& ctx, uint32_t v) {
  const RP* rp = rowptr<RP>(ctx);
  return rp[v + 1] > rp[v];
}

// gnz[b] = 1 if class b has a member with a non-empty row (gnz cleared for
// b < k by the caller).
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_live_class_nz(Ctx ctx) {
  for (uint32_t p = blockIdx.x * kBlock + threadIdx.x; p < ctx.n; p += gridDim.x * kBlock)
    if (row_nonempty<RP>(ctx, ctx.perm[p])) ctx.gnz[ctx.ids[p]] = 1;
}

__device__ __forceinline__ bool class_live(const Ctx& ctx, uint32_t b) {
  return ctx.cstart[b + 1] - ctx.cstart[b] >= 2 && ctx.gnz[b];
}

// gl[b] = 1, go[b] = size for live classes b < k, else 0 (scanned next).
__global__ void __launch_bounds__(kBlock) k_live_class_vals(Ctx ctx) {
  const uint32_t k = ctx.st->k;
  for (uint32_t b = blockIdx.x * kBlock + threadIdx.x; b < k; b += gridDim.x * kBlock) {
    const bool live = class_live(ctx, b);
    ctx.gl[b] = live ? 1u : 0u;
    ctx.go[b] = live ? ctx.cstart[b + 1] - ctx.cstart[b] : 0u;
  }
}

// Members of the live classes in colour order, with their row spans (into
// the '2' buffers, made current by k_live_commit).
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_live_build(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  for (uint32_t p = blockIdx.x * kBlock + threadIdx.x; p < ctx.n; p += gridDim.x * kBlock) {
    const uint32_t b = ctx.ids[p], v = ctx.perm[p];
    const bool live = class_live(ctx, b);
    if (!live) {
      if (ctx.pos) ctx.pos[v] = 0xFFFFFFFFu;
      continue;
    }
    const uint64_t r0 = rp[v], r1 = rp[v + 1];
    const uint32_t s = ctx.cstart[b];
    const uint32_t j = ctx.gl[b], q = ctx.go[b] + (p - s);
    if (ctx.pos) ctx.pos[v] = q;
    ctx.lperm2[q] = v;
    ctx.qcls2[q] = j;
    ctx.rs2[q] = r0;
    ctx.rl2[q] = (uint32_t)(r1 - r0);
    if (p == s) {
      ctx.lcold2[j] = b;
      ctx.loff2[j] = ctx.go[b];
      ctx.llen2[j] = ctx.cstart[b + 1] - s;
    }
  }
}

// ---------------------------------------------------------------------------
// One round
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(kBlock) k_live_load(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t nl = st->nl;
  for (uint32_t q = blockIdx.x * kBlock + threadIdx.x; q < nl; q += gridDim.x * kBlock) {
    ctx.keys[q] = ctx.rl[q] ? ctx.z[ctx.lperm[q]] : 0ull;
  }
}

// Sort work lists of the live classes (every one has >= 2 members); keys are
// materialised in 'keys'.
__global__ void __launch_bounds__(kBlock) k_live_segments(Ctx ctx) {
  DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t nlive = st->n_live;
  const uint32_t stride = gridDim.x * kBlock;
  for (uint32_t j0 = blockIdx.x * kBlock; j0 < nlive; j0 += stride) {
    const uint32_t j = j0 + threadIdx.x;
    uint32_t s = 0, len = 0;
    if (j < nlive) {
      s = ctx.loff[j];
      len = ctx.llen[j];
    }
    // 0 pico, 1 tiny, 2 mid, 3 small, 4 big, 5 none
    const uint32_t kind = len < 2 ? 5u
                          : len <= kPicoMax ? 0u
                          : len <= kTinyMax ? 1u
                          : len <= kMidMax ? 2u
                          : len <= kSmallMax ? 3u : 4u;
    const uint32_t at =
        block_append4(kind, &st->n_pico, &st->n_tiny, &st->n_msort, &st->n_small);
    if (kind == 0) ctx.tiny_list[ctx.max_small - 1 - at] = make_uint2(s, len | kMatBit);
    else if (kind == 1) ctx.tiny_list[at] = make_uint2(s, len | kMatBit);
    else if (kind == 2) ctx.small_list[ctx.max_sm - 1 - at] = make_uint2(s, len | kMatBit);
    else if (kind == 3) ctx.small_list[at] = make_uint2(s, len | kMatBit);
    else if (kind == 4) big_append(ctx, 0, s, len);
  }
}

// Classes and keys of positions q0 - 1 .. q0 + 4 (q0 a multiple of 4, q0 <
// nl; entries at or beyond nl, and before 0, are placeholders), from which
// the sub-class flags of q0 .. q0 + 4 follow: a sub-class starts at q when q
// is a class's first position or the key changes.
struct FlagWindow {
  uint32_t c[6];
  uint64_t k[6];
  __device__ __forceinline__ void load(const Ctx& ctx, uint32_t q0, uint32_t nl) {
    load4(ctx.qcls, q0, nl, c + 1);
    load4(ctx.keys, q0, nl, k + 1);
    c[0] = q0 ? ctx.qcls[q0 - 1] : 0xFFFFFFFFu;
    k[0] = q0 ? ctx.keys[q0 - 1] : 0ull;
    c[5] = q0 + 4 < nl ? ctx.qcls[q0 + 4] : 0xFFFFFFFFu;
    k[5] = q0 + 4 < nl ? ctx.keys[q0 + 4] : 0ull;
  }
  // flag of q0 + u, u <= 4 (q0 + u < nl)
  __device__ __forceinline__ uint32_t flag(uint32_t q0, int u) const {
    return (q0 + u == 0 || c[u + 1] != c[u] || k[u + 1] != k[u]) ? 1u : 0u;
  }
};

__global__ void __launch_bounds__(kBlock) k_live_scan_part(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done) return;
  uint32_t lo, hi;
  xscan_range(st->nl, blockIdx.x, gridDim.x, &lo, &hi);
  uint32_t s = 0;
  for (uint32_t q0 = lo + kScanItems * threadIdx.x; q0 < hi; q0 += kScanStep) {
    FlagWindow w;
    w.load(ctx, q0, st->nl);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (q0 + u < hi) s += w.flag(q0, u);
  }
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t tot;
  block_excl_scan(s, sh, &tot);
  if (threadIdx.x == 0) ctx.scan_part[blockIdx.x] = tot;
}

// Every block: its offset among the block sums and their total, the number
// of sub-classes of the live classes, nsub (block 0 records it with k_new =
// k + nsub - n_live and nosplit when no class split).  Then ids[q] =
// sub-class of q; per
// sub-class g: first position, end, and whether it holds a non-empty row:
// its key is non-zero (gnz), or a member with key 0 has one (its image
// happens to be 0; nz0f).
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_live_scan_final(Ctx ctx) {
  DevState* st = ctx.st;
  if (st->done) return;
  static_assert(kScanBlocks <= 4 * kBlock, "block sums summed by one block");
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t nsub;
  uint32_t run = block_part_prefix(ctx.scan_part, gridDim.x, blockIdx.x, sh, &nsub);
  const uint32_t nlive = st->n_live;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->nsub = nsub;
    st->k_new = st->k + nsub - nlive;
    st->nosplit = nsub == nlive ? 1u : 0u;
    st->split_any = nsub == nlive ? 0u : 1u;
    st->shift_big = 0;
  }
  if (nsub == nlive) return;
  const uint32_t nl = st->nl;
  uint32_t lo, hi;
  xscan_range(nl, blockIdx.x, gridDim.x, &lo, &hi);
  for (uint32_t base = lo; base < hi; base += kScanStep) {
    const uint32_t q0 = base + kScanItems * threadIdx.x;
    FlagWindow w;
    uint32_t f[5] = {0, 0, 0, 0, 0}, local = 0;
    if (q0 < hi) {
      w.load(ctx, q0, nl);
#pragma unroll
      for (int u = 0; u < 5; ++u) f[u] = q0 + u < nl ? w.flag(q0, u) : 0u;
#pragma unroll
      for (int u = 0; u < 4; ++u) local += q0 + u < hi ? f[u] : 0u;
    }
    uint32_t tot;
    // sub-class of q0 - 1: the ones of q0 .. q0 + u are added on the way
    uint32_t g = run + block_excl_scan(local, sh, &tot) - 1;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t q = q0 + u;
      if (q >= hi) break;
      g += f[u];
      ctx.ids[q] = g;
      const uint64_t key = w.k[u + 1];
      if (f[u]) {
        ctx.gstart[g] = q;
        ctx.gnz[g] = key != 0 ? 1 : 0;
      }
      if (key == 0 && row_nonempty<RP>(ctx, ctx.lperm[q])) ctx.nz0f[g] = 1;
      if (q + 1 == nl || f[u + 1]) ctx.gend[g] = q + 1;
    }
    run += tot;
  }
}

// The live sub-classes (gl[g] = 1, go[g] = size; scanned next), with the
// key-0 flags folded into gnz; and the classes that split: (old colour,
// extra sub-classes) in colour order (the live classes are in colour order,
// and each chunk of kBlock of them finds its place in the list by a chained
// scan of the chunks' split counts).  The block of the last chunk records
// the number of splits and whether they need the per-colour shift table.
// The first nscan blocks take the sub-classes in the ranges of the scan of
// gl and go that follows (k_xscan_final over nscan blocks), four consecutive
// ones per thread and step, and leave that scan its block sums in scan_part,
// in place of a launch of k_xscan_part.
__global__ void __launch_bounds__(kBlock) k_live_subs_splits(Ctx ctx, uint32_t nscan) {
  DevState* st = ctx.st;
  if (st->done || st->nosplit) return;
  const uint32_t ns = st->nsub;
  __shared__ uint32_t sh[kBlock / kWave];
  if (blockIdx.x < nscan) {
    uint32_t lo, hi;
    xscan_range(ns, blockIdx.x, nscan, &lo, &hi);
    uint32_t sa = 0, sb = 0;
    for (uint32_t g0 = lo + kScanItems * threadIdx.x; g0 < hi; g0 += kScanStep) {
#pragma unroll
      for (uint32_t u = 0; u < kScanItems; ++u) {
        const uint32_t g = g0 + u;
        if (g >= hi) break;
        bool nz = ctx.gnz[g] != 0;
        if (ctx.nz0f[g]) {
          ctx.nz0f[g] = 0;
          ctx.gnz[g] = 1;
          nz = true;
        }
        const uint32_t len = ctx.gend[g] - ctx.gstart[g];
        const bool live = len >= 2 && nz;
        ctx.gl[g] = live ? 1u : 0u;
        ctx.go[g] = live ? len : 0u;
        sa += live ? 1u : 0u;
        sb += live ? len : 0u;
      }
    }
    uint32_t ta, tb;
    block_excl_scan(sa, sh, &ta);
    block_excl_scan(sb, sh, &tb);
    if (threadIdx.x == 0) {
      ctx.scan_part[blockIdx.x] = ta;
      ctx.scan_part[nscan + blockIdx.x] = tb;
    }
  }
  __shared__ uint32_t sh1;
  const uint32_t nlive = st->n_live;
  const uint32_t nchunks = (nlive + kBlock - 1) / kBlock;
  const uint32_t epoch = chain_epoch(st->round, kChainSplits);
  // the first min(grid, nchunks) blocks take the chunks by ticket: one
  // ticket each when the grid covers them, so that no more atomics than
  // chunks hit the counter
  if (blockIdx.x >= nchunks) return;
  const bool one = gridDim.x >= nchunks;
  for (bool first = true; first || !one; first = false) {
    const uint32_t c = chain_ticket(&st->tickets[kChainSplits], &sh1);
    if (c >= nchunks) break;
    const uint32_t j = c * kBlock + threadIdx.x;
    uint32_t extra = 0;
    if (j < nlive) {
      const uint32_t s = ctx.loff[j];
      extra = ctx.ids[s + ctx.llen[j] - 1] - ctx.ids[s];
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan(extra > 0 ? 1u : 0u, sh, &tot);
    const uint32_t base = chain_prefix(ctx.desc, c, tot, epoch, ctx.chain_spins, st, &sh1);
    if (extra > 0) ctx.split[base + ex] = make_uint2(ctx.lcold[j], extra);
    if (j < nlive) ctx.lsplit[j] = extra > 0 ? 1 : 0;
    if (c == nchunks - 1 && threadIdx.x == 0) {
      st->n_split = base + tot;
      st->shift_big = base + tot > kShiftLds ? 1u : 0u;
    }
  }
}

// More than kShiftLds splits: shift table over all colours, shift[b] =
// extras of the split classes below b (delta at the split colours, then an
// exclusive scan).
__global__ void __launch_bounds__(kBlock) k_shift_clear(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done || !st->shift_big) return;
  const uint32_t k = st->k;
  for (uint32_t b = blockIdx.x * kBlock + threadIdx.x; b < k; b += gridDim.x * kBlock)
    ctx.shift[b] = 0;
}

__global__ void __launch_bounds__(kBlock) k_shift_scatter(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done || !st->shift_big) return;
  const uint32_t S = st->n_split;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < S; i += gridDim.x * kBlock) {
    const uint2 e = ctx.split[i];
    ctx.shift[e.x] = e.y;
  }
}

// New colour of every node: b + shift(b).  Members of the classes that
// split are rewritten by k_live_emit afterwards.  Four nodes per thread and
// step (16-byte accesses when the colour array allows).
// With the split list in LDS, shift(b) = cumulative extras of the last split
// colour below b.  With more than kShiftDirect splits the colours [0, k) are
// cut into kShiftBuckets ranges of 2^bsh colours, and bidx[t] = first split
// whose colour is in range t or above, so the search for b only visits the
// splits of b's own range; with fewer, the search spans all of them.
constexpr uint32_t kShiftBuckets = 1024;
constexpr uint32_t kShiftDirect = 256;

// The last split colour < b is at an index in [l, h], and scol[l] < b.
__device__ __forceinline__ uint32_t shift_lds(const uint32_t* scol, const uint32_t* scum,
                                              uint32_t l, uint32_t h, uint32_t b) {
  while (l < h) {
    const uint32_t mid = (l + h + 1) >> 1;
    if (scol[mid] < b) l = mid; else h = mid - 1;
  }
  return scum[l];
}

// halt != 0 (a device-driven round, which launched no kernels for the
// shift table): splits that need the table halt the device instead, for the
// host to build it and finish the round.
__global__ void __launch_bounds__(kBlock) k_shift_apply(Ctx ctx, int halt) {
  DevState* st = ctx.st;
  if (st->done || st->nosplit) return;
  const uint32_t S = st->n_split;
  const uint32_t n = ctx.n;
  const bool big = st->shift_big != 0;
  if (big && halt) {
    if (blockIdx.x == 0 && threadIdx.x == 0) st->done = kHaltedShift;
    return;
  }
  __shared__ uint32_t scol[kShiftLds];
  __shared__ uint32_t scum[kShiftLds];
  __shared__ uint32_t bidx[kShiftBuckets + 1];
  __shared__ uint32_t sh[kBlock / kWave];
  // every colour is below k: (k - 1) >> bsh < kShiftBuckets
  uint32_t bsh = 0;
  while (((st->k - 1) >> bsh) >= kShiftBuckets) ++bsh;
  const bool direct = S <= kShiftDirect;
  if (!big) {
    // the split list (S >= 1 when a class split), in colour order, with the
    // extras replaced by their inclusive prefix sums: each thread takes
    // kPer consecutive entries
    constexpr uint32_t kPer = kShiftLds / kBlock;
    const uint32_t t0 = threadIdx.x * kPer;
    uint32_t v[kPer], loc = 0;
#pragma unroll
    for (uint32_t u = 0; u < kPer; ++u) {
      v[u] = 0;
      if (t0 + u < S) {
        const uint2 e = ctx.split[t0 + u];
        scol[t0 + u] = e.x;
        v[u] = e.y;
      }
      loc += v[u];
    }
    uint32_t tot;
    uint32_t run = block_excl_scan(loc, sh, &tot);
#pragma unroll
    for (uint32_t u = 0; u < kPer; ++u)
      if (t0 + u < S) {
        run += v[u];
        scum[t0 + u] = run;
      }
    __syncthreads();
    for (uint32_t t = threadIdx.x; !direct && t <= kShiftBuckets; t += kBlock) {
      const uint64_t v = (uint64_t)t << bsh;
      uint32_t lo = 0, hi = S;
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (scol[mid] < v) lo = mid + 1; else hi = mid;
      }
      bidx[t] = lo;
    }
    __syncthreads();
  }
  const uint32_t first = big ? 0u : scol[0];
  auto moved = [&](uint32_t b) -> uint32_t {
    if (big) return b + ctx.shift[b];
    if (b <= first) return b;
    // b > scol[0]: the last split colour below b
    uint32_t l = 0, h = S - 1;
    if (!direct) {
      const uint32_t t = min(b >> bsh, kShiftBuckets - 1);
      const uint32_t lo = bidx[t], hi = bidx[t + 1];
      l = lo > 0 ? lo - 1 : 0;  // scol[lo - 1] < t << bsh <= b
      h = max(hi, l + 1) - 1;   // scol[hi] >= (t + 1) << bsh > b
    }
    return b + shift_lds(scol, scum, l, h, b);
  };
  const uint32_t tid = blockIdx.x * kBlock + threadIdx.x, stride = gridDim.x * kBlock;
  uint32_t done4 = 0;
  if (((uintptr_t)ctx.c & 15) == 0) {
    // with at least four groups of four colours per thread: four per step
    // (i, i + stride, ...), loaded together
    constexpr uint32_t kStep = 4;
    uint4* c4 = (uint4*)ctx.c;
    const uint32_t n4 = n / 4;
    const uint32_t step = (uint64_t)n4 >= (uint64_t)kStep * stride ? kStep : 1u;
    for (uint32_t i0 = tid; i0 < n4; i0 += step * stride) {
      uint4 a[kStep];
#pragma unroll
      for (uint32_t u = 0; u < kStep; ++u) {
        const uint32_t i = i0 + u * stride;
        if (u < step && i < n4) a[u] = c4[i];
      }
#pragma unroll
      for (uint32_t u = 0; u < kStep; ++u) {
        const uint32_t i = i0 + u * stride;
        if (u >= step || i >= n4) break;
        uint4 r;
        r.x = moved(a[u].x);
        r.y = moved(a[u].y);
        r.z = moved(a[u].z);
        r.w = moved(a[u].w);
        if (r.x != a[u].x || r.y != a[u].y || r.z != a[u].z || r.w != a[u].w) c4[i] = r;
      }
    }
    done4 = n4 * 4;
  }
  for (uint32_t i = done4 + tid; i < n; i += stride) {
    const uint32_t b = ctx.c[i];
    const uint32_t r = moved(b);
    if (r != b) ctx.c[i] = r;
  }
}

// Exact new colours of the members of classes that split, and the next live
// classes ('2' buffers).
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_live_emit(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done || st->nosplit) return;
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t nl = st->nl;
  for (uint32_t q = blockIdx.x * kBlock + threadIdx.x; q < nl; q += gridDim.x * kBlock) {
    const uint32_t v = ctx.lperm[q];
    const uint32_t j = ctx.qcls[q];
    const uint32_t g = ctx.ids[q];
    const uint32_t id = ctx.lcold[j] + g - j;
    const uint32_t gs = ctx.gstart[g];
    const uint32_t len = ctx.gend[g] - gs;
    uint64_t r0;
    uint32_t rlen;
    if (ctx.lsplit[j]) {
      ctx.c[v] = id;
      if (!(len >= 2 && ctx.gnz[g])) {
        if (ctx.pos) ctx.pos[v] = 0xFFFFFFFFu;  // its class leaves the live set
        continue;
      }
      r0 = rp[v];
      rlen = (uint32_t)(rp[v + 1] - r0);
    } else {
      // a class that did not split: its colour was moved by k_shift_apply,
      // it stays live (it has a non-empty row) and was not reordered
      r0 = ctx.rs[q];
      rlen = ctx.rl[q];
    }
    const uint32_t jn = ctx.gl[g], off = ctx.go[g];
    const uint32_t q2 = off + (q - gs);
    if (ctx.pos) ctx.pos[v] = q2;
    ctx.lperm2[q2] = v;
    ctx.qcls2[q2] = jn;
    ctx.rs2[q2] = r0;
    ctx.rl2[q2] = rlen;
    if (q == gs) {
      ctx.lcold2[jn] = id;
      ctx.loff2[jn] = off;
      ctx.llen2[jn] = len;
    }
  }
}

// The '2' buffers become current (their counts n_live2, nl2 are taken over
// by k_round_end / k_live_adopt).
__global__ void __launch_bounds__(kBlock) k_live_commit(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done || st->nosplit) return;
  const uint32_t nl = st->nl2, nlive = st->n_live2;
  const uint32_t tid = blockIdx.x * kBlock + threadIdx.x, stride = gridDim.x * kBlock;
  for (uint32_t q = tid; q < nl; q += stride) {
    ctx.lperm[q] = ctx.lperm2[q];
    ctx.qcls[q] = ctx.qcls2[q];
    ctx.rs[q] = ctx.rs2[q];
    ctx.rl[q] = ctx.rl2[q];
  }
  for (uint32_t j = tid; j < nlive; j += stride) {
    ctx.lcold[j] = ctx.lcold2[j];
    ctx.loff[j] = ctx.loff2[j];
    ctx.llen[j] = ctx.llen2[j];
  }
}

// After the set-up: the live counts take effect.
__global__ void k_live_adopt(Ctx ctx) {
  DevState* st = ctx.st;
  st->n_live = st->n_live2;
  st->nl = st->nl2;
}

// End of a live round (one thread): the colour count, round counter,
// termination and new live counts; the per-round counters are cleared.  No
// argument depends on the round, so the launch can be replayed.
__global__ void k_live_round_end(Ctx ctx) {
  DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t kn = st->k_new;
  st->round += 1;
  if (st->nosplit) {
    st->done = 1;
  } else {
    if (st->round >= st->max_rounds) st->done = 2;
    st->n_live = st->n_live2;
    st->nl = st->nl2;
  }
  st->k = kn;
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

}  // namespace wl
