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
  for (uint32_t i = lo + threadIdx.x; i < hi; i += kBlock) {
    int b = row_bin((uint64_t)(rp[i + 1] - rp[i]));
    cnt[b]++;
  }
  __shared__ uint32_t sh[kNumBins];
  if (threadIdx.x < kNumBins) sh[threadIdx.x] = 0;
  __syncthreads();
  for (int b = 0; b < kNumBins; ++b)
    if (cnt[b]) atomicAdd(&sh[b], cnt[b]);
  __syncthreads();
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

template <typename RP>
__global__ void __launch_bounds__(kBlock) k_bins_fill(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t n = ctx.n;
  const uint32_t per = (n + gridDim.x - 1) / gridDim.x;
  const uint32_t lo = min(n, blockIdx.x * per), hi = min(n, lo + per);
  __shared__ uint32_t sh[kBlock / kWave];
  uint32_t run[kNumBins];
  for (int b = 0; b < kNumBins; ++b)
    run[b] = ctx.st->bin_start[b] + ctx.bin_part[b * gridDim.x + blockIdx.x];
  for (uint32_t base = lo; base < hi; base += kBlock) {
    uint32_t i = base + threadIdx.x;
    int mybin = -1;
    if (i < hi) mybin = row_bin((uint64_t)(rp[i + 1] - rp[i]));
    for (int b = 0; b < kNumBins; ++b) {
      uint32_t tot;
      uint32_t ex = block_excl_scan(mybin == b ? 1u : 0u, sh, &tot);
      if (mybin == b) ctx.rows[run[b] + ex] = i;
      run[b] += tot;
    }
  }
}

// One block: chunk list of the heavy rows (bin 3).
template <typename RP>
__global__ void __launch_bounds__(kBlock) k_heavy_prep(Ctx ctx) {
  const RP* rp = rowptr<RP>(ctx);
  __shared__ uint32_t sh[kBlock / kWave];
  const uint32_t nh = ctx.st->bin_cnt[3];
  const uint32_t* list = ctx.rows + ctx.st->bin_start[3];
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nh; base += kBlock) {
    uint32_t h = base + threadIdx.x;
    uint32_t nc = 0, row = 0;
    uint64_t b0 = 0, e0 = 0;
    if (h < nh) {
      row = list[h];
      b0 = rp[row];
      e0 = rp[row + 1];
      nc = (uint32_t)((e0 - b0 + kHeavyChunk - 1) / kHeavyChunk);
    }
    uint32_t tot;
    uint32_t ex = block_excl_scan(nc, sh, &tot);
    for (uint32_t t = 0; t < nc; ++t) {
      HeavyChunk ch;
      ch.beg = b0 + (uint64_t)t * kHeavyChunk;
      ch.end = min(e0, ch.beg + kHeavyChunk);
      ch.row = row;
      ch.h = h;
      ctx.chunks[carry + ex + t] = ch;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) ctx.st->n_chunks = carry;
  for (uint32_t h = threadIdx.x; h < 2 * nh; h += kBlock) ctx.hacc[h] = 0;
}

// ---------------------------------------------------------------------------
// Per-node random values x_i = W(seed, round, c_i).
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(kBlock) k_weights(Ctx ctx) {
  if (ctx.st->done) return;
  const uint64_t key = round_key(ctx.st->seed, ctx.st->round);
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n;
       i += gridDim.x * kBlock)
    ctx.x[i] = color_weight(key, ctx.c[i]);
}

// ---------------------------------------------------------------------------
// SpMV kernels
// ---------------------------------------------------------------------------

template <int G, typename RP, bool W>
__global__ void __launch_bounds__(kBlock) k_spmv_group(Ctx ctx, int bin) {
  if (ctx.st->done) return;
  const RP* rp = rowptr<RP>(ctx);
  const uint32_t cnt = ctx.st->bin_cnt[bin];
  const uint32_t* list = ctx.rows + ctx.st->bin_start[bin];
  const uint32_t sub = threadIdx.x % G;
  const uint32_t ngroups = gridDim.x * (kBlock / G);
  for (uint32_t t = (blockIdx.x * kBlock + threadIdx.x) / G; t < cnt;
       t += ngroups) {
    const uint32_t row = list[t];
    if (!ctx.act[row]) continue;
    const uint64_t beg = rp[row], end = rp[row + 1];
    Acc96 a{0, 0};
    for (uint64_t e = beg + sub; e < end; e += G) {
      uint64_t v = ctx.x[ctx.col[e]];
      if (W) v = mul_small_fold(ctx.wgt[e], v);
      acc_add(a, v);
    }
    uint64_t r = group_sum_p<G>(acc_reduce(a));
    if (sub == 0) ctx.z[row] = r;
  }
}

template <typename RP, bool W>
__global__ void __launch_bounds__(kBlock) k_spmv_heavy(Ctx ctx) {
  if (ctx.st->done) return;
  const uint32_t nch = ctx.st->n_chunks;
  const int lane = lane_id();
  const uint32_t nwaves = gridDim.x * (kBlock / kWave);
  for (uint32_t t = (blockIdx.x * kBlock + threadIdx.x) / kWave; t < nch;
       t += nwaves) {
    const HeavyChunk ch = ctx.chunks[t];
    if (!ctx.act[ch.row]) continue;
    Acc96 a{0, 0};
    for (uint64_t e = ch.beg + lane; e < ch.end; e += kWave) {
      uint64_t v = ctx.x[ctx.col[e]];
      if (W) v = mul_small_fold(ctx.wgt[e], v);
      acc_add(a, v);
    }
    uint64_t r = group_sum_p<kWave>(acc_reduce(a));
    if (lane == 0) {
      atomicAdd(&ctx.hacc[2 * ch.h], (unsigned long long)(r & 0xFFFFFFFFull));
      atomicAdd(&ctx.hacc[2 * ch.h + 1], (unsigned long long)(r >> 32));
    }
  }
}

// z of the heavy rows = hi * 2^32 + lo (mod p); clears the accumulators.
__global__ void __launch_bounds__(kBlock) k_spmv_heavy_fin(Ctx ctx) {
  if (ctx.st->done) return;
  const uint32_t nh = ctx.st->bin_cnt[3];
  const uint32_t* list = ctx.rows + ctx.st->bin_start[3];
  for (uint32_t h = blockIdx.x * kBlock + threadIdx.x; h < nh;
       h += gridDim.x * kBlock) {
    const uint32_t row = list[h];
    if (ctx.act[row]) {
      uint64_t lo = ctx.hacc[2 * h], hi = fold61(ctx.hacc[2 * h + 1]);
      // hi * 2^32 = (hi mod 2^29) * 2^32 + (hi >> 29) * 2^61, 2^61 = 1.
      uint64_t t = ((hi & 0x1FFFFFFFull) << 32) + (hi >> 29);
      ctx.z[row] = addp(fold61(t), fold61(lo));
    }
    ctx.hacc[2 * h] = 0;
    ctx.hacc[2 * h + 1] = 0;
  }
}

}  // namespace wl
