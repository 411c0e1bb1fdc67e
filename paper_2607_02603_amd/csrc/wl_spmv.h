// Step "z = A w" of Algorithm 1 (Section 4.1): CSR SpMV in F_p.
//
// Rows are scheduled once per call into four length bins (wl_ctx.h):
// groups of 4, 16 or 64 lanes per row, and rows longer than kHeavyChunk cut
// into chunks of one wave each.  A row is skipped when its colour class is a
// singleton: its image cannot split anything (a singleton pair is unique
// whatever z is), so the rank-based relabel does not need it.
//
// Every lane accumulates exactly in 96 bits and folds once; lanes and chunks
// are combined with modular additions, which are associative, so the result
// does not depend on the schedule.
#pragma once
#include "wl_block.h"

namespace wl {

template <typename RP>
__device__ __forceinline__ const RP* rowptr(const Ctx& c);
template <>
__device__ __forceinline__ const uint32_t* rowptr<uint32_t>(const Ctx& c) {
  return c.rp32;
}
template <>
__device__ __forceinline__ const uint64_t* rowptr<uint64_t>(const Ctx& c) {
  return c.rp64;
}

// ---------------------------------------------------------------------------
// Schedule: rows of each bin, in node order.
// ---------------------------------------------------------------------------

template <typename RP>
__global__ void __launch_bounds__(kBlock) k_bins_count(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t n = ctx.n;
  const uint32_t per = (n + gridDim.x - 1) / gridDim.x;
  const uint32_t lo = min(n, blockIdx.x * per), hi = min(n, lo + per);
  uint32_t cnt[kNumBins] = {0, 0, 0, 0};
  uint64_t mx = 0;
  // four rows per thread and step (i, i + kBlock, ...), loaded together
  constexpr uint32_t kStep = 4;
  for (uint32_t i0 = lo + threadIdx.x; i0 < hi; i0 += kStep * kBlock) {
    uint64_t len[kStep];
#pragma unroll
    for (uint32_t u = 0; u < kStep; ++u) {
      const uint32_t i = i0 + u * kBlock;
      len[u] = i < hi ? (uint64_t)(rp[i + 1] - rp[i]) : ~0ull;
    }
#pragma unroll
    for (uint32_t u = 0; u < kStep; ++u)
      if (len[u] != ~0ull) {
        cnt[row_bin(len[u])]++;
        mx = len[u] > mx ? len[u] : mx;
      }
  }
  __shared__ uint32_t sh[kNumBins];
  __shared__ uint32_t smx;
  if (threadIdx.x < kNumBins) sh[threadIdx.x] = 0;
  if (threadIdx.x == 0) smx = 0;
  __syncthreads();
  for (int b = 0; b < kNumBins; ++b)
    if (cnt[b]) atomicAdd(&sh[b], cnt[b]);
  atomicMax(&smx, (uint32_t)(mx < 0xFFFFFFFFull ? mx : 0xFFFFFFFFull));
  __syncthreads();
  if (threadIdx.x == 0 && smx) atomicMax(&ctx.st->max_deg, smx);
  if (threadIdx.x < kNumBins)
    ctx.bin_part[threadIdx.x * gridDim.x + blockIdx.x] = sh[threadIdx.x];
}

// One block: exclusive scan of the per-block bin counts, bin totals/starts.
__global__ void __launch_bounds__(kBlock) k_bins_scan(Ctx ctx, uint32_t nblk) {
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t start = 0;
  for (int b = 0; b < kNumBins; ++b) {
    uint32_t carry = 0;
    uint32_t* part = ctx.bin_part + b * nblk;
    for (uint32_t base = 0; base < nblk; base += kBlock) {
      uint32_t i = base + threadIdx.x;
      uint32_t v = i < nblk ? part[i] : 0;
      uint32_t tot;
      uint32_t ex = block_excl_scan(v, sh, &tot);
      if (i < nblk) part[i] = carry + ex;
      carry += tot;
    }
    if (threadIdx.x == 0) {
      ctx.st->bin_cnt[b] = carry;
      ctx.st->bin_start[b] = start;
    }
    start += carry;
  }
}

// HEAVY: only the heavy rows' list (bin 3) is written (the incremental
// rounds use nothing else of the static schedule).
template <typename RP, bool HEAVY>
__global__ void __launch_bounds__(kBlock) k_bins_fill(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t n = ctx.n;
  const uint32_t per = (n + gridDim.x - 1) / gridDim.x;
  const uint32_t lo = min(n, blockIdx.x * per), hi = min(n, lo + per);
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t run[kNumBins];
  for (int b = 0; b < kNumBins; ++b)
    run[b] = ctx.st->bin_start[b] + ctx.bin_part[b * gridDim.x + blockIdx.x];
  // four groups of kBlock rows per step, their row lengths loaded together;
  // the groups are listed in order, so every list stays in node order
  constexpr uint32_t kStep = 4;
  for (uint32_t base = lo; base < hi; base += kStep * kBlock) {
    int mb[kStep];
    bool heavy = false;
#pragma unroll
    for (uint32_t u = 0; u < kStep; ++u) {
      const uint32_t i = base + u * kBlock + threadIdx.x;
      mb[u] = i < hi ? row_bin((uint64_t)(rp[i + 1] - rp[i])) : -1;
      heavy = heavy || mb[u] == 3;
    }
    // heavy rows are rare: a step without one needs no scan
    if (HEAVY && !__syncthreads_or(heavy)) continue;
#pragma unroll
    for (uint32_t u = 0; u < kStep; ++u) {
      const uint32_t i = base + u * kBlock + threadIdx.x;
      for (int b = HEAVY ? 3 : 0; b < kNumBins; ++b) {
        uint32_t tot;
        uint32_t ex = block_excl_scan(mb[u] == b ? 1u : 0u, sh, &tot);
        if (mb[u] == b) ctx.rows[run[b] + ex] = i;
        run[b] += tot;
      }
    }
  }
}

// Chunk list of the heavy rows (bin 3), in three launches: chunks per block
// of heavy rows, exclusive scan of the block totals, fill.
__device__ __forceinline__ void heavy_range(uint32_t nh, uint32_t b, uint32_t nblk,
                                            uint32_t* lo, uint32_t* hi) {
  const uint32_t per = (nh + nblk - 1) / nblk;
  *lo = min(nh, b * per);
  *hi = min(nh, *lo + per);
}

template <typename RP>
__device__ __forceinline__ uint32_t heavy_chunks_of(const Ctx& ctx, uint32_t row) {
  const RP* rp = rowptr<RP>(ctx);
  return (uint32_t)((rp[row + 1] - rp[row] + kHeavyChunk - 1) / kHeavyChunk);
}

template <typename RP>
__global__ void __launch_bounds__(kBlock) k_heavy_count(Ctx ctx) {
  const uint32_t nh = ctx.st->bin_cnt[3];
  const uint32_t* list = ctx.rows + ctx.st->bin_start[3];
  uint32_t lo, hi;
  heavy_range(nh, blockIdx.x, gridDim.x, &lo, &hi);
  uint32_t c = 0;
  for (uint32_t h = lo + threadIdx.x; h < hi; h += kBlock)
    c += heavy_chunks_of<RP>(ctx, list[h]);
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t tot;
  block_excl_scan(c, sh, &tot);
  if (threadIdx.x == 0) ctx.scan_part[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(kBlock) k_heavy_scan(Ctx ctx, uint32_t nblk) {
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nblk; base += kBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nblk ? ctx.scan_part[i] : 0;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(v, sh, &tot);
    if (i < nblk) ctx.scan_part[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) ctx.st->n_chunks = carry;
}

template <typename RP>
__global__ void __launch_bounds__(kBlock) k_heavy_fill(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t nh = ctx.st->bin_cnt[3];
  const uint32_t* list = ctx.rows + ctx.st->bin_start[3];
  uint32_t lo, hi;
  heavy_range(nh, blockIdx.x, gridDim.x, &lo, &hi);
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t carry = ctx.scan_part[blockIdx.x];
  for (uint32_t base = lo; base < hi; base += kBlock) {
    const uint32_t h = base + threadIdx.x;
    uint32_t nc = 0, row = 0;
    uint64_t b0 = 0, e0 = 0;
    if (h < hi) {
      row = list[h];
      b0 = rp[row];
      e0 = rp[row + 1];
      nc = (uint32_t)((e0 - b0 + kHeavyChunk - 1) / kHeavyChunk);
      ctx.hacc[2 * h] = 0;
      ctx.hacc[2 * h + 1] = 0;
      ctx.hcnt[h] = 0;
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan(nc, sh, &tot);
    for (uint32_t t = 0; t < nc; ++t) {
      HeavyChunk ch;
      ch.beg = b0 + (uint64_t)t * kHeavyChunk;
      ch.len = (uint32_t)(min(e0, ch.beg + kHeavyChunk) - ch.beg);
      ch.row = row;
      ch.h = h;
      ch.nc = nc;
      ctx.chunks[carry + ex + t] = ch;
    }
    carry += tot;
  }
}

// ---------------------------------------------------------------------------
// SpMV: one launch per round.  Each lane keeps U independent gathers in
// flight per iteration.
// ---------------------------------------------------------------------------

// Where the SpMV reads the random value of a neighbour j:
//   kGatherC   W(c[j]) computed from the colour (any number of colours)
//   kGather16  tbl[c16[j]], c16 = colour  (k <= 65535: 2 bytes per node)
//   kGather8   tbl[c8[j]],  c8  = colour  (k <= 255:   1 byte per node)
// The compact colour arrays shrink the randomly gathered footprint 4-8x; the
// table of k values stays in cache.
enum GatherMode { kGatherC = 0, kGather16 = 1, kGather8 = 2 };

__host__ __device__ __forceinline__ int gather_mode(uint32_t k) {
  return k <= 255 ? kGather8 : (k <= kTableMax ? kGather16 : kGatherC);
}

template <int M>
__device__ __forceinline__ uint64_t gather_value(const Ctx& ctx, uint32_t j,
                                                 uint64_t rkey) {
  if (ctx.batch) {
    const uint32_t jl = j - ctx.ext_lo;
    if (jl >= ctx.n) return color_weight64(rkey, (1ull << 32) + j, ctx.ring);
    j = jl;
  }
  if (M == kGather16) return ctx.wtab[ctx.c16[j]];
  if (M == kGather8) return ctx.wtab[ctx.c8[j]];
  return color_weight(rkey, ctx.c[j], ctx.ring);
}

template <int U, bool W, int M>
__device__ __forceinline__ void accumulate(const Ctx& ctx, Acc96& a, uint64_t e0,
                                           uint64_t end, uint32_t stride,
                                           uint64_t rkey) {
  uint32_t j[U];
  bool ok[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint64_t e = e0 + (uint64_t)u * stride;
    ok[u] = e < end;
    j[u] = ok[u] ? (ctx.nt_stream ? __builtin_nontemporal_load(ctx.col + e) : ctx.col[e])
                 : 0u;
  }
  uint64_t v[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    v[u] = ok[u] ? gather_value<M>(ctx, j[u], rkey) : 0ull;
    if (W && ok[u]) v[u] = mul_small_q(ctx.wgt[e0 + (uint64_t)u * stride], v[u], ctx.ring);
  }
#pragma unroll
  for (int u = 0; u < U; ++u) acc_add(a, v[u]);
}

template <int G, int U, typename RP, bool W, int M>
__device__ __forceinline__ void spmv_rows(const Ctx& ctx, int bin, uint32_t bid,
                                          uint32_t nblk, uint64_t rkey) {
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t cnt = ctx.st->bin_cnt[bin];
  const uint32_t* list = ctx.rows + ctx.st->bin_start[bin];
  const uint32_t sub = threadIdx.x % G;
  const uint32_t gpb = kBlock / G;
  const uint32_t ngroups = nblk * gpb;
  for (uint32_t t = bid * gpb + threadIdx.x / G; t < cnt; t += ngroups) {
    const uint32_t row = list[t];
    if (!ctx.act[row]) continue;
    const uint64_t beg = rp[row], end = rp[row + 1];
    Acc96 a{0, 0};
    for (uint64_t e0 = beg + sub; e0 < end; e0 += (uint64_t)G * U)
      accumulate<U, W, M>(ctx, a, e0, end, G, rkey);
    const uint64_t r = group_sum_q<G>(acc_value(a, ctx.ring), ctx.ring);
    if (sub == 0) ctx.z[row] = r;
  }
}

template <bool W, int M>
__device__ __forceinline__ void spmv_heavy(const Ctx& ctx, uint32_t bid,
                                           uint32_t nblk, uint64_t rkey) {
  const uint32_t nch = ctx.st->n_chunks;
  const int lane = lane_id();
  const uint32_t nwaves = nblk * (kBlock / kWave);
  for (uint32_t t = bid * (kBlock / kWave) + threadIdx.x / kWave; t < nch;
       t += nwaves) {
    const HeavyChunk ch = ctx.chunks[t];
    if (!ctx.act[ch.row]) continue;
    Acc96 a{0, 0};
    const uint64_t end = ch.beg + ch.len;
    for (uint64_t e0 = ch.beg + lane; e0 < end; e0 += (uint64_t)kWave * 4)
      accumulate<4, W, M>(ctx, a, e0, end, kWave, rkey);
    const uint64_t r = group_sum_q<kWave>(acc_value(a, ctx.ring), ctx.ring);
    if (lane == 0) {
      // Partial sums of the row's chunks meet in two 64-bit accumulators
      // (low and high 32-bit halves of the chunk values); the chunk that
      // finishes last folds them into z and resets them for the next round.
      atomicAdd(&ctx.hacc[2 * ch.h], (unsigned long long)(r & 0xFFFFFFFFull));
      atomicAdd(&ctx.hacc[2 * ch.h + 1], (unsigned long long)(r >> 32));
      __threadfence();
      const uint32_t seen = atomicAdd(&ctx.hcnt[ch.h], 1u);
      if (seen == ch.nc - 1) {
        __threadfence();
        const uint64_t lo = atomicExch(&ctx.hacc[2 * ch.h], 0ull);
        const uint64_t hs = atomicExch(&ctx.hacc[2 * ch.h + 1], 0ull);
        atomicExch(&ctx.hcnt[ch.h], 0u);
        if (ctx.ring) {
          ctx.z[ch.row] = lo + (hs << 32);  // mod 2^64
        } else {
          // hi * 2^32 = (hi mod 2^29) * 2^32 + (hi >> 29) * 2^61, 2^61 = 1.
          const uint64_t hi = fold61(hs);
          const uint64_t t2 = ((hi & 0x1FFFFFFFull) << 32) + (hi >> 29);
          ctx.z[ch.row] = addp(fold61(t2), fold61(lo));
        }
      }
    }
  }
}

template <typename RP, bool W, int M>
__device__ __forceinline__ void spmv_body(const Ctx& ctx, const SpmvGrid& g) {
  const uint64_t rkey = round_key(ctx.st->seed, ctx.st->round);
  const uint32_t b = blockIdx.x;
  if (b < g.heavy)
    spmv_heavy<W, M>(ctx, b, g.heavy, rkey);
  else if (b < g.b2)
    spmv_rows<64, 4, RP, W, M>(ctx, 2, b - g.heavy, g.b2 - g.heavy, rkey);
  else if (b < g.b1)
    spmv_rows<16, 4, RP, W, M>(ctx, 1, b - g.b2, g.b1 - g.b2, rkey);
  else
    spmv_rows<4, 2, RP, W, M>(ctx, 0, b - g.b1, g.b0 - g.b1, rkey);
}

template <typename RP, bool W, int M>
__global__ void __launch_bounds__(kBlock) k_spmv(Ctx ctx, SpmvGrid g) {
  if (ctx.st->done) return;
  spmv_body<RP, W, M>(ctx, g);
}

// ---------------------------------------------------------------------------
// Image of the live rows, by position q of lperm: the row of position q
// starts at rs[q] and has rl[q] entries (kept with the member list, so no
// per-node lookups).  Rows of at most kShortRow entries take one lane each;
// longer ones are queued for one wave each (k_spmv_mid), and rows longer
// than kHeavyChunk go through the static heavy chunks (which write z;
// k_live_heavy_fix moves those images to the keys).  Empty rows have key 0.
// ---------------------------------------------------------------------------

constexpr uint32_t kShortRow = 16;

template <bool W, int M>
__device__ __forceinline__ void spmv_q_body(const Ctx& ctx) {
  DevState* st = ctx.st;
  const uint64_t rkey = round_key(st->seed, st->round);
  const uint32_t nl = st->nl;
  __shared__ uint32_t sh[kBlock / kWave];
  __shared__ uint32_t base_sh;
  for (uint32_t q0 = blockIdx.x * kBlock; q0 < nl; q0 += gridDim.x * kBlock) {
    const uint32_t q = q0 + threadIdx.x;
    uint32_t len = 0;
    uint64_t beg = 0;
    if (q < nl) {
      len = ctx.rl[q];
      beg = ctx.rs[q];
    }
    const bool heavy = len > kHeavyChunk;
    const bool mid = len > kShortRow && !heavy;
    const uint32_t am = block_append(mid, &st->n_mid, sh, &base_sh);
    if (mid) ctx.midq[am] = q;
    const uint32_t ah = block_append(heavy, &st->n_hlive, sh, &base_sh);
    if (heavy) ctx.hq[ah] = q;
    if (q < nl && !mid && !heavy) {
      Acc96 a{0, 0};
      for (uint32_t t0 = 0; t0 < len; t0 += 4) {
        uint32_t j[4];
        bool ok[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          ok[u] = t0 + u < len;
          j[u] = ok[u] ? ctx.col[beg + t0 + u] : 0u;
        }
        uint64_t v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          v[u] = ok[u] ? gather_value<M>(ctx, j[u], rkey) : 0ull;
          if (W && ok[u]) v[u] = mul_small_q(ctx.wgt[beg + t0 + u], v[u], ctx.ring);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) acc_add(a, v[u]);
      }
      ctx.keys[q] = acc_value(a, ctx.ring);
    }
  }
}

// The gathering image of the live rows taken in node order, for graphs
// whose rows have at most kShortRow entries (one lane per row, nothing to
// queue): pos[v] is v's position among the live rows (~0 if none), so
// consecutive lanes read consecutive rows and, on graphs with locality,
// nearby colours.
template <typename RP, bool W>
__global__ void __launch_bounds__(kBlock) k_spmv_node(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done) return;
  const uint64_t rkey = round_key(st->seed, st->round);
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t n = ctx.n;
  for (uint32_t v = blockIdx.x * kBlock + threadIdx.x; v < n; v += gridDim.x * kBlock) {
    const uint32_t q = ctx.pos[v];
    if (q == 0xFFFFFFFFu) continue;
    const uint64_t beg = rp[v];
    const uint32_t len = (uint32_t)(rp[v + 1] - beg);
    Acc96 a{0, 0};
    for (uint32_t t0 = 0; t0 < len; t0 += 4) {
      uint32_t j[4];
      bool ok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ok[u] = t0 + u < len;
        j[u] = ok[u] ? ctx.col[beg + t0 + u] : 0u;
      }
      uint64_t val[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        val[u] = ok[u] ? gather_value<kGatherC>(ctx, j[u], rkey) : 0ull;
        if (W && ok[u]) val[u] = mul_small_q(ctx.wgt[beg + t0 + u], val[u], ctx.ring);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) acc_add(a, val[u]);
    }
    ctx.keys[q] = acc_value(a, ctx.ring);
  }
}

// The live rounds compute every neighbour's value from its colour
// (kGatherC): the compact colour tables would cost a pass over all n
// colours per round, and their lookups are random reads.
template <bool W>
__global__ void __launch_bounds__(kBlock) k_spmv_q(Ctx ctx) {
  if (ctx.st->done) return;
  spmv_q_body<W, kGatherC>(ctx);
}

// Blocks [0, heavy): the static heavy chunks (rows whose act flag is set by
// k_heavy_set); the rest: one wave per queued row.
template <bool W, int M>
__device__ __forceinline__ void spmv_mid_body(const Ctx& ctx, uint32_t heavy) {
  const uint64_t rkey = round_key(ctx.st->seed, ctx.st->round);
  if (blockIdx.x < heavy) {
    spmv_heavy<W, M>(ctx, blockIdx.x, heavy, rkey);
    return;
  }
  const uint32_t cnt = ctx.st->n_mid;
  const uint32_t lane = lane_id();
  const uint32_t nwaves = (gridDim.x - heavy) * (kBlock / kWave);
  for (uint32_t t = (blockIdx.x - heavy) * (kBlock / kWave) + threadIdx.x / kWave; t < cnt;
       t += nwaves) {
    const uint32_t q = ctx.midq[t];
    const uint64_t beg = ctx.rs[q], end = beg + ctx.rl[q];
    Acc96 a{0, 0};
    for (uint64_t e0 = beg + lane; e0 < end; e0 += (uint64_t)kWave * 4)
      accumulate<4, W, M>(ctx, a, e0, end, kWave, rkey);
    const uint64_t r = group_sum_q<kWave>(acc_value(a, ctx.ring), ctx.ring);
    if (lane == 0) ctx.keys[q] = r;
  }
}

template <bool W>
__global__ void __launch_bounds__(kBlock) k_spmv_mid(Ctx ctx, uint32_t heavy) {
  if (ctx.st->done) return;
  spmv_mid_body<W, kGatherC>(ctx, heavy);
}

// act of the heavy rows for the static chunks: 0 for every heavy row, then 1
// for those of live classes (listed by k_spmv_q).
__global__ void __launch_bounds__(kBlock) k_heavy_clear(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t nh = st->bin_cnt[3];
  const uint32_t* list = ctx.rows + st->bin_start[3];
  for (uint32_t t = blockIdx.x * kBlock + threadIdx.x; t < nh; t += gridDim.x * kBlock)
    ctx.act[list[t]] = 0;
}

__global__ void __launch_bounds__(kBlock) k_heavy_set(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t cnt = st->n_hlive;
  for (uint32_t t = blockIdx.x * kBlock + threadIdx.x; t < cnt; t += gridDim.x * kBlock)
    ctx.act[ctx.lperm[ctx.hq[t]]] = 1;
}

// Heavy live rows: their images (written to z by the chunks) into keys.
__global__ void __launch_bounds__(kBlock) k_live_heavy_fix(Ctx ctx) {
  const DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t cnt = st->n_hlive;
  for (uint32_t t = blockIdx.x * kBlock + threadIdx.x; t < cnt; t += gridDim.x * kBlock) {
    const uint32_t q = ctx.hq[t];
    ctx.keys[q] = ctx.z[ctx.lperm[q]];
  }
}

// Rows and entries of the live rows (diagnostics, and the choice of the
// propagation-blocking image): st->act_entries, and with 'work' the
// diagnostic counters.
__global__ void __launch_bounds__(kBlock) k_live_count(Ctx ctx, int work) {
  const DevState* st = ctx.st;
  if (st->done) return;
  const uint32_t nl = st->nl;
  unsigned long long rows = 0, ents = 0;
  for (uint32_t q = blockIdx.x * kBlock + threadIdx.x; q < nl; q += gridDim.x * kBlock) {
    const uint32_t l = ctx.rl[q];
    rows += l ? 1 : 0;
    ents += l;
  }
  __shared__ unsigned long long sr[kBlock], se[kBlock];
  sr[threadIdx.x] = rows;
  se[threadIdx.x] = ents;
  __syncthreads();
  for (int o = kBlock / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      sr[threadIdx.x] += sr[threadIdx.x + o];
      se[threadIdx.x] += se[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0 && se[0]) {
    if (work) {
      atomicAdd(&ctx.st->work[kImgGather][0], sr[0]);
      atomicAdd(&ctx.st->work[kImgGather][1], se[0]);
    } else {
      atomicAdd(&ctx.st->act_entries, se[0]);
    }
  }
}

// One colour and unit weights: every x_j is the same w, so
// z_i = deg_i * w exactly, without touching col_idx.
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_spmv_uniform(Ctx ctx) {
  if (ctx.st->done) return;
  const RP* rp = rowptr<RP>(ctx);
  const uint64_t w0 = color_weight(round_key(ctx.st->seed, ctx.st->round), 0, ctx.ring);
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock)
    ctx.z[i] = mul_int_q(rp[i + 1] - rp[i], w0, ctx.ring);
}

// Per-round random values for the gather: compact colour array plus the
// table of the k colour values (k <= 65535); with more colours the SpMV
// computes each value from the neighbour's colour.
// mode < 0: chosen from the colour count on the device.
__device__ __forceinline__ void gather_prep_body(const Ctx& ctx, int mode, uint32_t k,
                                                 uint64_t key) {
  const uint32_t tid = blockIdx.x * kBlock + threadIdx.x;
  const uint32_t stride = gridDim.x * kBlock;
  if (mode == kGatherC) return;
  for (uint32_t b = tid; b < k; b += stride) ctx.wtab[b] = color_weight(key, b, ctx.ring);
  if (mode == kGather16)
    for (uint32_t i = tid; i < ctx.n; i += stride) ctx.c16[i] = (uint16_t)ctx.c[i];
  else
    for (uint32_t i = tid; i < ctx.n; i += stride) ctx.c8[i] = (uint8_t)ctx.c[i];
}

__global__ void __launch_bounds__(kBlock) k_gather_prep(Ctx ctx, int mode) {
  if (ctx.st->done) return;
  const uint32_t k = ctx.st->k;
  gather_prep_body(ctx, mode < 0 ? gather_mode(k) : mode, k,
                   round_key(ctx.st->seed, ctx.st->round));
}

// Diagnostics: rows and entries the next image launch of 'kind' reads (all
// of them when 'all' is set: the propagation-blocking image reads every
// entry); otherwise the rows with act set.
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_count_work(Ctx ctx, int kind, int all) {
  if (ctx.st->done) return;
  const RP* rp = rowptr<RP>(ctx);
  unsigned long long rows = 0, ents = 0;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock)
    if (all || ctx.act[i]) {
      rows += 1;
      ents += rp[i + 1] - rp[i];
    }
  __shared__ unsigned long long sr[kBlock], se[kBlock];
  sr[threadIdx.x] = rows;
  se[threadIdx.x] = ents;
  __syncthreads();
  for (int o = kBlock / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      sr[threadIdx.x] += sr[threadIdx.x + o];
      se[threadIdx.x] += se[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0 && sr[0]) {
    atomicAdd(&ctx.st->work[kind][0], sr[0]);
    atomicAdd(&ctx.st->work[kind][1], se[0]);
  }
}


// Entries of the rows whose image is needed this round, added to
// st->act_entries (cleared by k_round_begin).
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_count_active(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  unsigned long long ents = 0;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n; i += gridDim.x * kBlock)
    if (ctx.act[i]) ents += rp[i + 1] - rp[i];
  __shared__ unsigned long long se[kBlock];
  se[threadIdx.x] = ents;
  __syncthreads();
  for (int o = kBlock / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) se[threadIdx.x] += se[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0 && se[0]) atomicAdd(&ctx.st->act_entries, se[0]);
}

}  // namespace wl
