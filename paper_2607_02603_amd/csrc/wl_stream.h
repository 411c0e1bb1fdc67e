// Step "z = A w" of Algorithm 1 (Section 4.1) for a graph whose entries stay
// in host memory.  Every round the host packs the rows whose image is needed
// (act set, at least one entry) into segments of at most kSegMax entries and
// copies them to the device chunk by chunk; the colours, the images and the
// whole relabel stay on the device.  A row longer than kSegMax is cut into
// several segments whose partial sums are folded into z by k_stream_fold; a
// row whose segments reach into the next chunk is continued there (the fold
// adds to the z already written).
#pragma once
#include "wl_host.h"
#include "wl_spmv.h"

namespace wl {

// One chunk on the device.
struct StreamChunk {
  const uint32_t* node;  // per segment: node id | kSegPartial for a cut row
  const uint64_t* off;   // nseg + 1 entry offsets into col / wt
  const uint32_t* col;
  const uint32_t* wt;    // NULL: every entry weighs 1
  uint64_t* part;        // per segment: partial sum of a cut row
  const StreamFold* fold;  // per cut row of the chunk (wl_host.h)
  uint32_t nseg, nfold;
};

template <bool W, int M>
__device__ __forceinline__ void stream_seg_body(const Ctx& ctx, const StreamChunk& ch) {
  const uint64_t rkey = round_key(ctx.st->seed, ctx.st->round);
  const uint32_t lane = lane_id();
  const uint32_t nwaves = gridDim.x * (kBlock / kWave);
  for (uint32_t t = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; t < ch.nseg;
       t += nwaves) {
    const uint64_t beg = ch.off[t], end = ch.off[t + 1];
    Acc96 a{0, 0};
    for (uint64_t e0 = beg + lane; e0 < end; e0 += (uint64_t)kWave * 4) {
      uint32_t j[4];
      bool ok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint64_t e = e0 + (uint64_t)u * kWave;
        ok[u] = e < end;
        j[u] = ok[u] ? ch.col[e] : 0u;
      }
      uint64_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[u] = ok[u] ? gather_value<M>(ctx, j[u], rkey) : 0ull;
        if (W && ok[u]) v[u] = mul_small_q(ch.wt[e0 + (uint64_t)u * kWave], v[u], ctx.ring);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) acc_add(a, v[u]);
    }
    const uint64_t r = group_sum_q<kWave>(acc_value(a, ctx.ring), ctx.ring);
    if (lane == 0) {
      const uint32_t nd = ch.node[t];
      if (nd & kSegPartial)
        ch.part[t] = r;
      else
        ctx.z[nd] = r;
    }
  }
}

// One wave per segment.
template <bool W>
__global__ void __launch_bounds__(kBlock) k_stream_seg(Ctx ctx, StreamChunk ch) {
  if (ctx.st->done) return;
  const int mode = gather_mode(ctx.st->k);
  if (mode == kGather8)
    stream_seg_body<W, kGather8>(ctx, ch);
  else if (mode == kGather16)
    stream_seg_body<W, kGather16>(ctx, ch);
  else
    stream_seg_body<W, kGatherC>(ctx, ch);
}

// One thread per cut row of the chunk: z = (z if continued) + its partials.
__global__ void __launch_bounds__(kBlock) k_stream_fold(Ctx ctx, StreamChunk ch) {
  if (ctx.st->done) return;
  for (uint32_t f = blockIdx.x * kBlock + threadIdx.x; f < ch.nfold; f += gridDim.x * kBlock) {
    const StreamFold d = ch.fold[f];
    uint64_t s = d.add ? ctx.z[d.node] : 0ull;
    for (uint32_t t = 0; t < d.count; ++t) s = add_q(s, ch.part[d.first + t], ctx.ring);
    ctx.z[d.node] = s;
  }
}

// One colour, unit weights: z_i = deg_i * w without the entries.
__global__ void __launch_bounds__(kBlock) k_stream_uniform(Ctx ctx, const uint32_t* deg) {
  if (ctx.st->done) return;
  const uint64_t w0 = color_weight(round_key(ctx.st->seed, ctx.st->round), 0, ctx.ring);
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < ctx.n; i += gridDim.x * kBlock)
    ctx.z[i] = mul_int_q(deg[i], w0, ctx.ring);
}

__global__ void __launch_bounds__(kBlock) k_zero_u64(uint64_t* p, uint64_t n) {
  for (uint64_t i = blockIdx.x * (uint64_t)kBlock + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * kBlock)
    p[i] = 0;
}

}  // namespace wl
