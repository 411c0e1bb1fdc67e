// Step "z = A w" of Algorithm 1 for a symmetric A by propagation blocking.
//
// The gathering SpMV reads one value per entry at a random node, which costs
// a whole cache line per entry on graphs whose node order has no locality.
// When A is symmetric, the rows that hold node j are exactly the entries of
// row j, so every row can instead send its colour to its neighbours, and the
// traffic can be made sequential by routing the messages through bins of
// destination rows:
//   pass 1  stream the CSR entries in order; each tile of kPbTile entries
//           turns them into records (destination row inside its bin, colour
//           of the source row), counting-sorts them by bin in LDS and writes
//           one run per bin, reserved with an atomic on the bin's cursor;
//   pass 2  only when there are more than kPbMaxBins fine bins: pass 1 used
//           coarse bins of 2^fbits fine bins each; every coarse bin is split
//           into its fine bins the same way (run offsets from atomics), one
//           tile of kPbTile2 records per workgroup, neighbouring workgroups
//           on different coarse bins so that their reservations on the
//           bins' cursors do not queue behind each other;
//   pass 3  one workgroup per fine bin of kPbFineRows rows, or per slice of
//           at most kPbSlice records of a larger one, adds W(colour) of its
//           records into per-row accumulators in LDS; single-slice bins
//           write z, the partial sums of the others are added by a last
//           kernel.
// For symmetric A, the records bound for rows [a, b) number rp[b] - rp[a],
// so every bin occupies the entry range of its rows in the CSR layout.  The
// accumulators are exact (two 64-bit sums of the 32-bit halves of canonical
// residues per row) and every sum is reduced mod p at the end, so the image
// does not depend on the order in which records arrive.
#pragma once
#include "wl_spmv.h"

namespace wl {

constexpr int kPbFineShift = 13;
constexpr uint32_t kPbFineRows = 1u << kPbFineShift;  // rows per fine bin
constexpr uint32_t kPbMaxBins = 256;                  // bins of pass 1
constexpr uint32_t kPbMaxFine = 512;                  // fine bins per coarse bin
constexpr uint32_t kPbTile = 8192;                    // entries per pass-1 tile
constexpr uint32_t kPbTile2 = 4096;                   // records per pass-2 tile
constexpr uint32_t kPbSlice = 1u << 20;               // records per pass-3 item
constexpr int kPbThreads = 256;                       // pass 2 and the plan
constexpr int kPb1Threads = 512;                      // pass 1
constexpr int kPbAccThreads = 1024;                   // pass 3
constexpr uint32_t kErrNotSymmetric = 16u;  // DevState::err bit
constexpr uint64_t kPbMinEntries = 1ull << 22;  // smaller graphs stay in cache

// Device-side counts of the plan (read by the host once per call).
struct PbCounts {
  uint32_t ntiles2;   // pass-2 tiles
  uint32_t nslices;   // pass-3 work items
  uint32_t nmulti;    // fine bins with several slices
  uint32_t mslices;   // slices of those bins
  uint32_t maxtiles2; // most pass-2 tiles of one coarse bin
};

struct PbCtx {
  uint32_t levels;     // 1: pass 1 writes fine bins; 2: coarse bins, then pass 2
  uint32_t shift1;     // log2 of the rows of a pass-1 bin
  uint32_t nb1;        // pass-1 bins
  uint32_t nfine;      // fine bins
  uint32_t fbits;      // log2 of the fine bins per coarse bin (levels == 2)
  uint32_t cbits;      // bits of the colour in a record
  uint64_t ntiles1;    // pass-1 tiles
  uint64_t* bstart1;   // nb1 + 1: first entry of the rows of each pass-1 bin
  uint64_t* bstartf;   // nfine + 1: the same for the fine bins
  uint32_t* rec1;      // pass-1 records (coarse bins; levels == 2)
  uint32_t* rec2;      // fine-bin records
  uint32_t* tile_row;  // ntiles1: row that holds the first entry of each tile
  uint32_t* tile2_off; // nb1 + 1: pass-2 tiles before each coarse bin
  unsigned long long* cur1;  // nb1: write cursors of pass 1 (levels == 2)
  unsigned long long* cur2;  // nfine: write cursors of the fine bins
  uint32_t* slice_off;       // nfine + 1: pass-3 items before each fine bin
  uint32_t* mslice_off;      // nfine + 1: partial-sum slots before each bin
  uint32_t* mlist;           // fine bins with several slices
  uint64_t* part;            // partial images, kPbFineRows per slot
  PbCounts* cnt;
  // Non-null in the incremental round that follows the one-colour round:
  // the member-list position of every node (~0 outside the live classes).
  // Each live row's image then goes straight to its sort key (ctx.keys)
  // instead of to z in node order.
  const uint32_t* kpos;
};

template <typename RP>
__device__ __forceinline__ uint64_t rp_at(const Ctx& c, uint64_t i) {
  return (uint64_t)rowptr<RP>(c)[i];
}

// Start of the entry range of the rows [b << shift, ...) (clamped to n).
template <typename RP>
__device__ __forceinline__ uint64_t bin_start(const Ctx& c, uint64_t b, uint32_t shift) {
  const uint64_t r = b << shift;
  return rp_at<RP>(c, r < c.n ? r : c.n);
}

// Exclusive scan over a block of kPbThreads threads.
template <int T>
__device__ __forceinline__ uint32_t pb_block_scan(uint32_t v, uint32_t* sh, uint32_t* total) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  const uint32_t inc = wave_incl_scan(v);
  if (lane == kWave - 1) sh[wid] = inc;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < T / kWave; ++w) {
    const uint32_t s = sh[w];
    if (w < wid) base += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

// ---------------------------------------------------------------------------
// Plan (once per call; depends on the graph only)
// ---------------------------------------------------------------------------

template <typename RP>
__global__ void __launch_bounds__(kBlock) k_pb_bin_starts(Ctx ctx, PbCtx pb) {
  if (blockIdx.x == 0 && threadIdx.x == 0) pb.cnt->maxtiles2 = 0;
  for (uint32_t b = blockIdx.x * kBlock + threadIdx.x; b <= pb.nfine; b += gridDim.x * kBlock) {
    pb.bstartf[b] = bin_start<RP>(ctx, b, kPbFineShift);
    if (b <= pb.nb1) pb.bstart1[b] = bin_start<RP>(ctx, b, pb.shift1);
  }
}

// tile_row[t] = the row holding entry t * kPbTile.
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_pb_tile_rows(Ctx ctx, PbCtx pb) {
  for (uint32_t r = blockIdx.x * kBlock + threadIdx.x; r < ctx.n; r += gridDim.x * kBlock) {
    const uint64_t b = rp_at<RP>(ctx, r), e = rp_at<RP>(ctx, r + 1);
    if (e <= b) continue;
    for (uint64_t t = (b + kPbTile - 1) / kPbTile; t * kPbTile < e; ++t) pb.tile_row[t] = r;
  }
}

// One block: pass-2 tiles per coarse bin, pass-3 slices per fine bin, and
// the list of fine bins with several slices.
template <typename RP>
__global__ void __launch_bounds__(kPbThreads) k_pb_lists(Ctx ctx, PbCtx pb) {
  __shared__ uint32_t sh[kPbThreads / kWave];
  uint32_t carry = 0;
  if (pb.levels == 2) {
    for (uint32_t base = 0; base < pb.nb1; base += kPbThreads) {
      const uint32_t b = base + threadIdx.x;
      uint32_t nt = 0;
      if (b < pb.nb1) {
        const uint64_t sz = pb.bstart1[b + 1] - pb.bstart1[b];
        nt = (uint32_t)((sz + kPbTile2 - 1) / kPbTile2);
      }
      uint32_t tot;
      const uint32_t ex = pb_block_scan<kPbThreads>(nt, sh, &tot);
      if (b < pb.nb1) pb.tile2_off[b] = carry + ex;
      carry += tot;
      if (nt) atomicMax(&pb.cnt->maxtiles2, nt);
    }
    if (threadIdx.x == 0) {
      pb.tile2_off[pb.nb1] = carry;
      pb.cnt->ntiles2 = carry;
    }
  }
  uint32_t sc = 0, mc = 0, nm = 0;
  for (uint32_t base = 0; base < pb.nfine; base += kPbThreads) {
    const uint32_t f = base + threadIdx.x;
    uint32_t ns = 0;
    if (f < pb.nfine) {
      const uint64_t sz = pb.bstartf[f + 1] - pb.bstartf[f];
      ns = sz <= kPbSlice ? 1u : (uint32_t)((sz + kPbSlice - 1) / kPbSlice);
    }
    uint32_t tot, mtot, ntot;
    const uint32_t ex = pb_block_scan<kPbThreads>(ns, sh, &tot);
    const uint32_t mex = pb_block_scan<kPbThreads>(ns > 1 ? ns : 0u, sh, &mtot);
    const uint32_t nex = pb_block_scan<kPbThreads>(ns > 1 ? 1u : 0u, sh, &ntot);
    if (f < pb.nfine) {
      pb.slice_off[f] = sc + ex;
      pb.mslice_off[f] = mc + mex;
      if (ns > 1) pb.mlist[nm + nex] = f;
    }
    sc += tot;
    mc += mtot;
    nm += ntot;
  }
  if (threadIdx.x == 0) {
    pb.slice_off[pb.nfine] = sc;
    pb.mslice_off[pb.nfine] = mc;
    pb.cnt->nslices = sc;
    pb.cnt->nmulti = nm;
    pb.cnt->mslices = mc;
  }
}

// ---------------------------------------------------------------------------
// Passes 1 and 2 share the staging scheme: every record of a tile gets its
// rank inside its bin from an LDS atomic, the bins' run offsets come from a
// block scan and one cursor reservation per bin and tile, the records are
// staged in bin order in LDS and written out one slot per lane, consecutive
// over the lanes (staged slot s of bin b goes to dd[b] + s), so a wave's
// store covers whole runs.
// ---------------------------------------------------------------------------

constexpr long long kPbSkip = -(1ll << 62);  // dd of a run that is not written

template <int T, typename BT>
__device__ __forceinline__ void pb_write_out(const uint32_t* buf, const BT* sbin,
                                             const long long* dd, uint32_t cnt,
                                             uint32_t* out) {
  for (uint32_t s = threadIdx.x; s < cnt; s += T) {
    const long long o = dd[sbin[s]];
    if (o != kPbSkip) out[o + s] = buf[s];
  }
}

// Run offsets of a tile: hist[b] (records of bin b in the tile) becomes its
// exclusive prefix; one cursor reservation per non-empty bin; dd[b] = output
// index of staged slot 0 of bin b, or kPbSkip when the run would pass the
// bin's end (A is not symmetric: error bit, run dropped).  Bins
// [0, nbins) over the block's threads.  Contains __syncthreads().
__device__ __forceinline__ void pb_reserve(const Ctx& ctx, uint32_t* hist, long long* dd,
                                           uint32_t* sh, uint32_t nbins,
                                           unsigned long long* cur, const uint64_t* bstart) {
  uint32_t carry = 0;
  for (uint32_t b0 = 0; b0 < nbins; b0 += kPbThreads) {
    const uint32_t b = b0 + threadIdx.x;
    const uint32_t h = b < nbins ? hist[b] : 0u;
    uint32_t tot;
    const uint32_t ex = carry + pb_block_scan<kPbThreads>(h, sh, &tot);
    if (h) {
      const unsigned long long d = atomicAdd(&cur[b], (unsigned long long)h);
      if (d + h > bstart[b + 1]) {
        atomicOr(&ctx.st->err, kErrNotSymmetric);
        dd[b] = kPbSkip;
      } else {
        dd[b] = (long long)d - (long long)ex;
      }
    }
    if (b < nbins) hist[b] = ex;
    carry += tot;
  }
}

// ---------------------------------------------------------------------------
// Pass 1: CSR entries -> records in pass-1 bins
// ---------------------------------------------------------------------------

// Each tile of kPbTile entries, in the order that lets the latencies overlap:
//   1. the column indices (registers) and the first row-start data are
//      loaded together;
//   2. the first entry of every non-empty row starting in the tile is set
//      in a bit mask (one bit per entry, 1 KB) while every entry's bin is
//      counted (LDS adds whose returned old value is the entry's rank among
//      the tile's entries of that bin);
//   3. a block scan gives each bin's run offset in the tile and one cursor
//      reservation per bin is issued; while it is in flight, one wave turns
//      the mask into per-word prefix counts, every row start stores its
//      colour at its rank among the tile's row starts, and every entry finds
//      its row's colour from the number of row starts at or before it (the
//      row holding the tile's first entry has rank 0);
//   4. the reservations give each run's output offset (dd), the records are
//      staged by bin at their run's offset in the tile plus their rank, and
//      written out (pb_write_out).
// The packed bins of a thread's entries take 4 registers, their ranks 8.
// 512 threads, 4 waves per SIMD: two workgroups per CU (at most 128 VGPRs).
template <typename RP>
__global__ void __launch_bounds__(kPb1Threads, 4) k_pb_scatter1(Ctx ctx, PbCtx pb) {
  static_assert(kPbMaxBins <= kPb1Threads, "one thread per pass-1 bin in the reservation");
  if (ctx.st->done) return;
  constexpr uint32_t kRun = kPbTile / kPb1Threads;  // entries per thread
  constexpr uint32_t kGroups = kRun / 4;           // loads of 4 entries per thread
  constexpr uint32_t kWords = kPbTile / 32;         // words of the row-start mask
  static_assert(kWords <= kPb1Threads && kWords % kWave == 0, "mask words per thread");
  __shared__ __align__(16) uint32_t buf[kPbTile];  // row colours by rank, then staged records
  __shared__ __align__(16) uint8_t sbin[kPbTile];  // bin of each staged record
  __shared__ uint32_t bits[kWords];                // row starts of the tile
  __shared__ uint32_t wpre[kWords];                // row starts before each word
  __shared__ uint32_t hist[kPbMaxBins];
  __shared__ long long dd[kPbMaxBins];
  __shared__ uint32_t sh[kPb1Threads / kWave];
  const int lane = lane_id();
  const uint32_t mask1 = (1u << pb.shift1) - 1;
  const bool two = pb.levels == 2;
  uint32_t* out = two ? pb.rec1 : pb.rec2;
  unsigned long long* cur = two ? pb.cur1 : pb.cur2;
  const uint64_t* bstart = two ? pb.bstart1 : pb.bstartf;
  const uint4* col4 = (const uint4*)ctx.col;
  for (uint64_t t = blockIdx.x; t < pb.ntiles1; t += gridDim.x) {
    const uint64_t e0 = t * kPbTile, e1 = min(ctx.nnz, e0 + kPbTile);
    const uint32_t cnt = (uint32_t)(e1 - e0);
    const uint32_t j0 = pb.tile_row[t];
    const uint32_t jend = t + 1 < pb.ntiles1 ? pb.tile_row[t + 1] : ctx.n - 1;
    // 1. column indices: slot (k, u) holds entry 4 * (k * kPb1Threads + threadIdx.x) + u
    uint32_t cix[kRun];
    if (cnt == kPbTile) {
#pragma unroll
      for (uint32_t k = 0; k < kGroups; ++k) {
        const uint4 v = col4[(e0 >> 2) + k * kPb1Threads + threadIdx.x];
        cix[4 * k] = v.x;
        cix[4 * k + 1] = v.y;
        cix[4 * k + 2] = v.z;
        cix[4 * k + 3] = v.w;
      }
    } else {
#pragma unroll
      for (uint32_t k = 0; k < kGroups; ++k)
#pragma unroll
        for (uint32_t u = 0; u < 4; ++u) {
          const uint32_t q = 4 * (k * kPb1Threads + threadIdx.x) + u;
          cix[4 * k + u] = q < cnt ? ctx.col[e0 + q] : 0u;
        }
    }
    // the first row starting in the tile for this thread (rows j0 + 1 ..
    // jend start after e0; the row holding e0 is j0)
    const uint32_t r0 = j0 + 1 + threadIdx.x;
    uint64_t rb = 0, re = 0;
    uint32_t rc = 0;
    if (r0 <= jend) {
      rb = rp_at<RP>(ctx, r0);
      re = rp_at<RP>(ctx, r0 + 1);
      rc = ctx.c[r0];
    }
    const uint32_t c_first = ctx.c[j0];
    if (threadIdx.x < kWords) bits[threadIdx.x] = 0;
    if (threadIdx.x < kPbMaxBins) hist[threadIdx.x] = 0;
    __syncthreads();
    // 2. row starts into the mask; bins counted
    const bool first_starts = r0 <= jend && rb < e1 && re > rb;
    if (first_starts) atomicOr(&bits[(rb - e0) >> 5], 1u << ((rb - e0) & 31));
    for (uint32_t r = r0 + kPb1Threads; r <= jend; r += kPb1Threads) {
      const uint64_t b = rp_at<RP>(ctx, r);
      if (b < e1 && rp_at<RP>(ctx, r + 1) > b)
        atomicOr(&bits[(b - e0) >> 5], 1u << ((b - e0) & 31));
    }
    // the 4 bins of group k, one byte each (every byte value is a bin), and
    // bit 4k + u set when entry (k, u) has a record
    static_assert(kRun <= 32 && kPbMaxBins <= 256, "bins packed in bytes, validity in 32 bits");
    uint32_t bins[kGroups];
    uint32_t rk2[kRun / 2] = {};  // rank of each entry inside its bin in this tile, 16 bits
    uint32_t valid = 0;
#pragma unroll
    for (uint32_t k = 0; k < kGroups; ++k) {
      uint32_t w = 0;
#pragma unroll
      for (uint32_t u = 0; u < 4; ++u) {
        const uint32_t q = 4 * (k * kPb1Threads + threadIdx.x) + u;
        const uint32_t bn = cix[4 * k + u] >> pb.shift1;
        if (q < cnt) {
          if (bn < pb.nb1) {
            rk2[(4 * k + u) >> 1] |= atomicAdd(&hist[bn], 1u) << (16 * (u & 1));
            w |= bn << (8 * u);
            valid |= 1u << (4 * k + u);
          } else {  // a column >= n
            atomicOr(&ctx.st->err, kErrNotSymmetric);
          }
        }
      }
      bins[k] = w;
    }
    __syncthreads();
    // 3. run offsets and one cursor reservation per bin (thread = bin)
    const uint32_t h = threadIdx.x < kPbMaxBins ? hist[threadIdx.x] : 0u;
    uint32_t nrec;
    const uint32_t ex = pb_block_scan<kPb1Threads>(h, sh, &nrec);
    unsigned long long d = 0;
    if (h) d = atomicAdd(&cur[threadIdx.x], (unsigned long long)h);
    //    while it is in flight: row starts before each mask word (wave 0)
    if (threadIdx.x < kWave) {
      constexpr uint32_t kPer = kWords / kWave;
      uint32_t pc[kPer];
      uint32_t s = 0;
#pragma unroll
      for (uint32_t u = 0; u < kPer; ++u) {
        pc[u] = __popc(bits[lane * kPer + u]);
        s += pc[u];
      }
      uint32_t run = wave_incl_scan(s) - s;
#pragma unroll
      for (uint32_t u = 0; u < kPer; ++u) {
        wpre[lane * kPer + u] = run;
        run += pc[u];
      }
    }
    __syncthreads();
    //    the colour of every row start at its rank
    auto rank_below = [&](uint32_t pos) {  // row starts at positions < pos
      return wpre[pos >> 5] + __popc(bits[pos >> 5] & ((1u << (pos & 31)) - 1u));
    };
    if (first_starts) buf[rank_below((uint32_t)(rb - e0))] = rc;
    for (uint32_t r = r0 + kPb1Threads; r <= jend; r += kPb1Threads) {
      const uint64_t b = rp_at<RP>(ctx, r);
      if (b < e1 && rp_at<RP>(ctx, r + 1) > b) buf[rank_below((uint32_t)(b - e0))] = ctx.c[r];
    }
    __syncthreads();
    //    every entry's row colour, and the record
#pragma unroll
    for (uint32_t k = 0; k < kGroups; ++k) {
      const uint32_t q0 = 4 * (k * kPb1Threads + threadIdx.x);  // a multiple of 4
      const uint32_t wbits = bits[q0 >> 5], wbase = wpre[q0 >> 5];
      // row starts at positions <= q0; the next three positions lie in the
      // same mask word, and a set bit there starts the next row
      uint32_t rk = wbase + __popc(wbits & ((2u << (q0 & 31)) - 1u));
      uint32_t c = rk ? buf[rk - 1] : c_first;
#pragma unroll
      for (uint32_t u = 0; u < 4; ++u) {
        if (u > 0 && ((wbits >> ((q0 + u) & 31)) & 1u)) c = buf[rk++];
        const uint32_t i = cix[4 * k + u];
        cix[4 * k + u] = ((i & mask1) << pb.cbits) | c;  // the record
      }
    }
    // 4. output offsets of the runs (a bin without records in this tile
    //    gets kPbSkip, so no slot can reach a stale offset), then staging
    if (threadIdx.x < kPbMaxBins) {
      if (!h) {
        dd[threadIdx.x] = kPbSkip;
      } else if (d + h > bstart[threadIdx.x + 1]) {
        atomicOr(&ctx.st->err, kErrNotSymmetric);
        dd[threadIdx.x] = kPbSkip;
      } else {
        dd[threadIdx.x] = (long long)d - (long long)ex;
      }
    }
    __syncthreads();  // the row colours in buf are consumed; dd is complete
    if (threadIdx.x < kPbMaxBins) hist[threadIdx.x] = ex;
    __syncthreads();
#pragma unroll
    for (uint32_t k = 0; k < kGroups; ++k)
#pragma unroll
      for (uint32_t u = 0; u < 4; ++u)
        if (valid & (1u << (4 * k + u))) {
          const uint32_t bn = (bins[k] >> (8 * u)) & 0xFFu;
          const uint32_t slot = hist[bn] + ((rk2[(4 * k + u) >> 1] >> (16 * (u & 1))) & 0xFFFFu);
          buf[slot] = cix[4 * k + u];
          sbin[slot] = (uint8_t)bn;
        }
    __syncthreads();
    // only the staged records (a column >= n has none)
    pb_write_out<kPb1Threads, uint8_t>(buf, sbin, dd, nrec, out);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Pass 2: coarse bins -> fine bins
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(kBlock) k_pb_cursors(Ctx ctx, PbCtx pb) {
  if (ctx.st->done) return;
  for (uint32_t f = blockIdx.x * kBlock + threadIdx.x; f < pb.nfine; f += gridDim.x * kBlock) {
    pb.cur2[f] = pb.bstartf[f];
    if (f < pb.nb1) pb.cur1[f] = pb.bstart1[f];
  }
}

__global__ void __launch_bounds__(kPbThreads) k_pb_scatter2(Ctx ctx, PbCtx pb) {
  if (ctx.st->done || (ctx.st->err & kErrNotSymmetric)) return;
  __shared__ __align__(16) uint32_t buf[kPbTile2];
  __shared__ uint32_t hist[kPbMaxFine];
  __shared__ long long dd[kPbMaxFine];
  __shared__ uint32_t sh[kPbThreads / kWave];
  const uint32_t nf = 1u << pb.fbits;
  const uint32_t cmask = (1u << pb.cbits) - 1;
  constexpr uint32_t kPer = kPbTile2 / kPbThreads;
  // block v: tile v / nb1 of coarse bin v % nb1 (neighbouring blocks work on
  // different coarse bins, so their cursor reservations do not collide)
  const uint32_t cb = blockIdx.x % pb.nb1, r = blockIdx.x / pb.nb1;
  if (pb.tile2_off[cb] + r >= pb.tile2_off[cb + 1]) return;
  const uint64_t a0 = pb.bstart1[cb] + (uint64_t)r * kPbTile2;
  const uint32_t cnt = (uint32_t)(min(pb.bstart1[cb + 1], a0 + kPbTile2) - a0);
  uint32_t rec[kPer];
#pragma unroll
  for (uint32_t k = 0; k < kPer; ++k) {
    const uint32_t q = k * kPbThreads + threadIdx.x;
    rec[k] = q < cnt ? pb.rec1[a0 + q] : 0u;
  }
  const uint32_t nfb = min(nf, pb.nfine - (cb << pb.fbits));
  for (uint32_t b = threadIdx.x; b < nf; b += kPbThreads) hist[b] = 0;
  __syncthreads();
  uint32_t pk[kPer];
#pragma unroll
  for (uint32_t k = 0; k < kPer; ++k) {
    pk[k] = 0xFFFFFFFFu;
    if (k * kPbThreads + threadIdx.x < cnt) {
      const uint32_t local = rec[k] >> pb.cbits;
      const uint32_t b = min(local >> kPbFineShift, nfb - 1);
      pk[k] = (b << 16) | atomicAdd(&hist[b], 1u);
    }
  }
  __syncthreads();
  pb_reserve(ctx, hist, dd, sh, nfb, pb.cur2 + ((uint64_t)cb << pb.fbits),
             pb.bstartf + ((uint64_t)cb << pb.fbits));
  __syncthreads();
#pragma unroll
  for (uint32_t k = 0; k < kPer; ++k)
    if (pk[k] != 0xFFFFFFFFu) {
      const uint32_t b = pk[k] >> 16;
      buf[hist[b] + (pk[k] & 0xFFFF)] = rec[k];
    }
  __syncthreads();
  // the staged pass-1 records name their fine bin (the high bits of their
  // row), and are rewritten to the row inside it on the way out
  for (uint32_t s = threadIdx.x; s < cnt; s += kPbThreads) {
    const uint32_t r1 = buf[s];
    const uint32_t local = r1 >> pb.cbits;
    const long long o = dd[min(local >> kPbFineShift, nfb - 1)];
    if (o != kPbSkip)
      pb.rec2[o + s] = ((local & (kPbFineRows - 1)) << pb.cbits) | (r1 & cmask);
  }
}

// ---------------------------------------------------------------------------
// Pass 3: records of a fine bin -> z
// ---------------------------------------------------------------------------

// value = acc + carries * 2^64: mod p (2^64 = 8 mod p), or acc in Z/2^64
__device__ __forceinline__ uint64_t pb_reduce(uint64_t acc, uint32_t carries, uint32_t ring) {
  return ring ? acc : addp(fold61(acc), fold61((uint64_t)carries << 3));
}

// TBL: the k colour values sit in LDS (k <= kPbTableMax), else each record's
// value is computed from its colour.
constexpr uint32_t kPbTableMax = 4096;

// Per row an exact sum: a 64-bit accumulator (one atomic per record, whose
// returned old value shows a wrap past 2^64) and a count of such wraps.  In
// Z/2^64 the wraps are dropped (the accumulator is the sum mod 2^64).
__device__ __forceinline__ void pb_acc_add(unsigned long long* acc, uint32_t* wraps,
                                           uint32_t r, uint64_t v, uint32_t extra,
                                           uint32_t ring) {
  const unsigned long long old = atomicAdd(&acc[r], (unsigned long long)v);
  if (ring) return;
  const uint32_t w = extra + (old + v < old ? 1u : 0u);
  if (w) atomicAdd(&wraps[r], w);
}

template <typename RP, bool TBL>
__global__ void __launch_bounds__(kPbAccThreads) k_pb_accum(Ctx ctx, PbCtx pb) {
  if (ctx.st->done || (ctx.st->err & kErrNotSymmetric)) return;
  __shared__ unsigned long long acc[kPbFineRows];
  __shared__ uint32_t wraps[kPbFineRows];
  __shared__ uint64_t wtab[TBL ? kPbTableMax : 1];
  constexpr uint32_t kU = 4;  // records per thread per step, loaded together
  const uint64_t key = round_key(ctx.st->seed, ctx.st->round);
  const uint32_t cmask = (1u << pb.cbits) - 1;
  const uint32_t nitems = pb.cnt->nslices;
  if (TBL) {
    const uint32_t k = ctx.st->k;
    for (uint32_t b = threadIdx.x; b < k; b += kPbAccThreads)
      wtab[b] = color_weight(key, b, ctx.ring);
  }
  for (uint32_t t = blockIdx.x; t < nitems; t += gridDim.x) {
    uint32_t lo = 0, hi = pb.nfine - 1;  // fine bin: last f with slice_off[f] <= t
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) >> 1;
      if (pb.slice_off[mid] <= t) lo = mid; else hi = mid - 1;
    }
    const uint32_t f = lo;
    const uint32_t q = t - pb.slice_off[f];
    const uint32_t ns = pb.slice_off[f + 1] - pb.slice_off[f];
    const uint64_t b1 = pb.bstartf[f + 1];
    const uint64_t a = pb.bstartf[f] + (uint64_t)q * kPbSlice;
    const uint64_t e = ns == 1 ? b1 : min(b1, a + kPbSlice);
    for (uint32_t r = threadIdx.x; r < kPbFineRows; r += kPbAccThreads) {
      acc[r] = 0;
      wraps[r] = 0;
    }
    __syncthreads();
    uint32_t nxt[kU];
#pragma unroll
    for (uint32_t u = 0; u < kU; ++u) {
      const uint64_t p = a + u * kPbAccThreads + threadIdx.x;
      nxt[u] = p < e ? pb.rec2[p] : 0u;
    }
    for (uint64_t p0 = a; p0 < e; p0 += kU * kPbAccThreads) {
      uint32_t rv[kU];
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) rv[u] = nxt[u];
      // the next step's records are loaded while these are added
      const uint64_t p1 = p0 + kU * kPbAccThreads;
      if (p1 < e) {
#pragma unroll
        for (uint32_t u = 0; u < kU; ++u) {
          const uint64_t p = p1 + u * kPbAccThreads + threadIdx.x;
          nxt[u] = p < e ? pb.rec2[p] : 0u;
        }
      }
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        const bool ok = p0 + u * kPbAccThreads + threadIdx.x < e;
        const uint32_t local = (rv[u] >> pb.cbits) & (kPbFineRows - 1);
        const uint64_t w =
            ok ? (TBL ? wtab[rv[u] & cmask] : color_weight(key, rv[u] & cmask, ctx.ring))
               : 0ull;
        // every lane is active here: lane 0's row, without an LDS permute
        const uint32_t l0 = __builtin_amdgcn_readfirstlane(local);
        if (__all(!ok || local == l0)) {
          // the whole wave feeds one row (rows of high degree): add the 64
          // values exactly (low and high 32-bit halves) in registers first
          uint64_t sl = w & 0xFFFFFFFFull, sh2 = w >> 32;
#pragma unroll
          for (int off = kWave / 2; off > 0; off >>= 1) {
            sl += __shfl_xor(sl, off, kWave);
            sh2 += __shfl_xor(sh2, off, kWave);
          }
          if (lane_id() == 0 && (sl | sh2)) {
            // sl + sh2 * 2^32 as (64-bit part, multiples of 2^64)
            const uint64_t v = sl + (sh2 << 32);
            const uint32_t hi64 = (uint32_t)(sh2 >> 32) + (v < sl ? 1u : 0u);
            pb_acc_add(acc, wraps, l0, v, hi64, ctx.ring);
          }
        } else if (ok) {
          pb_acc_add(acc, wraps, local, w, 0, ctx.ring);
        }
      }
    }
    __syncthreads();
    const uint64_t row0 = (uint64_t)f << kPbFineShift;
    const uint32_t nrows = (uint32_t)min((uint64_t)kPbFineRows, (uint64_t)ctx.n - row0);
    if (ns == 1 && pb.kpos) {
      for (uint32_t r = threadIdx.x; r < nrows; r += kPbAccThreads) {
        const uint32_t q = pb.kpos[row0 + r];
        if (q != 0xFFFFFFFFu) ctx.keys[q] = pb_reduce(acc[r], wraps[r], ctx.ring);
      }
    } else if (ns == 1) {
      for (uint32_t r = threadIdx.x; r < nrows; r += kPbAccThreads)
        ctx.z[row0 + r] = pb_reduce(acc[r], wraps[r], ctx.ring);
    } else {
      uint64_t* part = pb.part + (uint64_t)(pb.mslice_off[f] + q) * kPbFineRows;
      for (uint32_t r = threadIdx.x; r < nrows; r += kPbAccThreads)
        part[r] = pb_reduce(acc[r], wraps[r], ctx.ring);
    }
    __syncthreads();
  }
}

// Bins with several slices: z = sum of the partial images.
__global__ void __launch_bounds__(kBlock) k_pb_combine(Ctx ctx, PbCtx pb) {
  if (ctx.st->done || (ctx.st->err & kErrNotSymmetric)) return;
  const uint32_t nm = pb.cnt->nmulti;
  const uint64_t total = (uint64_t)nm * kPbFineRows;
  for (uint64_t x = blockIdx.x * (uint64_t)kBlock + threadIdx.x; x < total;
       x += (uint64_t)gridDim.x * kBlock) {
    const uint32_t f = pb.mlist[x >> kPbFineShift];
    const uint32_t r = (uint32_t)(x & (kPbFineRows - 1));
    const uint64_t row = ((uint64_t)f << kPbFineShift) + r;
    if (row >= ctx.n) continue;
    const uint32_t s0 = pb.mslice_off[f], s1 = pb.mslice_off[f + 1];
    uint64_t z = 0;
    for (uint32_t s = s0; s < s1; ++s)
      z = add_q(z, pb.part[(uint64_t)s * kPbFineRows + r], ctx.ring);
    if (!pb.kpos) {
      ctx.z[row] = z;
    } else {
      const uint32_t q = pb.kpos[row];
      if (q != 0xFFFFFFFFu) ctx.keys[q] = z;
    }
  }
}

}  // namespace wl
