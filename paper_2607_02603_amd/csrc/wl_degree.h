// The round of Algorithm 1 (Section 4.1) that starts from a single colour on
// an unweighted graph, done without sorting the nodes.
//
// With one colour every neighbour carries the same random value w, so the
// image is z_i = deg_i * w (mod p) and the new colour of node i is the rank
// of deg_i * w among the distinct values d * w over the degrees d present
// (equal degrees give equal values; for w != 0 distinct degrees below p give
// distinct values, and the ranks are taken over the values themselves, so
// w = 0 is handled as well).  The work is a degree histogram, a sort of the
// distinct degrees' values (at most kDegRanks of them, in one workgroup), and
// a counting placement of the nodes of the new live classes, class after
// class, into the member list of the incremental rounds (wl_live.h).
// A graph with more distinct values than kDegRanks takes the general path.
#pragma once
#include "wl_live.h"

namespace wl {

constexpr uint32_t kDegRanks = 4096;  // distinct degrees handled in one workgroup
constexpr uint32_t kDegLds = 2048;    // degrees counted in LDS (larger: global atomics)
constexpr int kDegThreads = 1024;

// Scratch of the degree round (carved from the 'keys' region, 8 bytes per
// node: the degree table takes max_deg + 1 words, the rest sits behind it).
struct DegScratch {
  uint32_t* dcount;  // max_deg + 1: nodes per degree, then rank | live bit
  uint32_t* dlist;   // kDegRanks: present degrees (unordered)
  uint32_t* roff;    // kDegRanks: first member-list position of each rank
  uint32_t* rj;      // kDegRanks: live class index of each rank
  uint32_t* rdeg;    // kDegRanks: degree of each rank's nodes (kDegMixed: several)
  uint32_t* nd;      // number of present degrees (DevState::deg_nd)
};

// degree table entries after the ranking: rank | flags
constexpr uint32_t kDegLive = 0x80000000u;   // the rank is a live class
constexpr uint32_t kDegShared = 0x40000000u; // several degrees share the rank
constexpr uint32_t kDegRankMask = 0x3FFFFFFFu;
constexpr uint32_t kDegMixed = 0xFFFFFFFFu;

__device__ __forceinline__ uint32_t degree_of(const Ctx& ctx, uint32_t i, bool rp64) {
  return rp64 ? (uint32_t)(ctx.rp64[i + 1] - ctx.rp64[i]) : ctx.rp32[i + 1] - ctx.rp32[i];
}

__global__ void __launch_bounds__(kBlock) k_deg_clear(Ctx ctx, DegScratch d, uint32_t maxd) {
  for (uint32_t x = blockIdx.x * kBlock + threadIdx.x; x <= maxd; x += gridDim.x * kBlock)
    d.dcount[x] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) *d.nd = 0;
}

// The loops over the nodes below take kDegStep nodes per thread and step
// (i, i + kBlock, ...), their loads issued together.
constexpr uint32_t kDegStep = 4;

// Nodes per degree.
template <bool RP64>
__global__ void __launch_bounds__(kBlock) k_deg_hist(Ctx ctx, DegScratch d) {
  __shared__ uint32_t h[kDegLds];
  for (uint32_t x = threadIdx.x; x < kDegLds; x += kBlock) h[x] = 0;
  __syncthreads();
  const uint32_t stride = gridDim.x * kBlock * kDegStep;
  for (uint32_t i0 = blockIdx.x * kBlock * kDegStep + threadIdx.x; i0 < ctx.n; i0 += stride) {
    uint32_t g[kDegStep];
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) {
      const uint32_t i = i0 + u * kBlock;
      g[u] = i < ctx.n ? degree_of(ctx, i, RP64) : 0xFFFFFFFFu;
    }
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) {
      if (g[u] == 0xFFFFFFFFu) continue;
      if (g[u] < kDegLds)
        atomicAdd(&h[g[u]], 1u);
      else
        atomicAdd(&d.dcount[g[u]], 1u);
    }
  }
  __syncthreads();
  for (uint32_t x = threadIdx.x; x < kDegLds; x += kBlock)
    if (h[x]) atomicAdd(&d.dcount[x], h[x]);
}

// Present degrees, unordered (at most kDegRanks are kept; *nd counts all).
__global__ void __launch_bounds__(kBlock) k_deg_list(Ctx ctx, DegScratch d, uint32_t maxd) {
  __shared__ uint32_t sh[kBlock / kWave];
  __shared__ uint32_t base_sh;
  for (uint32_t x0 = blockIdx.x * kBlock; x0 <= maxd; x0 += gridDim.x * kBlock) {
    const uint32_t x = x0 + threadIdx.x;
    const bool present = x <= maxd && d.dcount[x] != 0;
    const uint32_t at = block_append(present, d.nd, sh, &base_sh);
    if (present && at < kDegRanks) d.dlist[at] = x;
  }
}

// One workgroup: values d * w of the present degrees, sorted; rank of every
// degree = number of distinct smaller values; per rank its node count and
// whether it forms a live class (>= 2 nodes, a non-empty row); live classes
// numbered in rank order with their member-list offsets.  Writes the live
// class table (in place) and the next round's counts, k_new and nosplit.
__global__ void __launch_bounds__(kDegThreads) k_deg_ranks(Ctx ctx, DegScratch d) {
  DevState* st = ctx.st;
  const uint32_t D = *d.nd;
  if (D > kDegRanks) return;  // the host takes the general path
  __shared__ unsigned long long key[kDegRanks];
  __shared__ uint32_t deg[kDegRanks];
  __shared__ uint32_t rk[kDegRanks];    // rank of sorted slot t
  __shared__ uint32_t wsum[kDegThreads / kWave];
  __shared__ uint32_t wsum2[kDegThreads / kWave];
  const uint64_t w = color_weight(round_key(st->seed, st->round), 0, ctx.ring);
  uint32_t P = 1;
  while (P < D) P <<= 1;
  for (uint32_t t = threadIdx.x; t < P; t += kDegThreads) {
    if (t < D) {
      const uint32_t g = d.dlist[t];
      deg[t] = g;
      key[t] = mul_int_q(g, w, ctx.ring);
    } else {
      deg[t] = 0xFFFFFFFFu;
      key[t] = ~0ull;
    }
  }
  __syncthreads();
  for (uint32_t kk = 2; kk <= P; kk <<= 1)
    for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < P; i += kDegThreads) {
        const uint32_t l = i ^ j;
        if (l > i) {
          const bool asc = (i & kk) == 0;
          const unsigned long long a = key[i], b = key[l];
          // ties broken by degree so the order is total
          const bool gt = a > b || (a == b && deg[i] > deg[l]);
          if (gt == asc) {
            key[i] = b;
            key[l] = a;
            const uint32_t tv = deg[i];
            deg[i] = deg[l];
            deg[l] = tv;
          }
        }
      }
      __syncthreads();
    }
  // rank of slot t = distinct keys before it (block scan of "new key" flags)
  constexpr uint32_t kPer = kDegRanks / kDegThreads;
  const uint32_t t0 = threadIdx.x * kPer;
  const int lane = lane_id(), wid = threadIdx.x / kWave;
  {
    uint32_t loc = 0;
#pragma unroll
    for (uint32_t u = 0; u < kPer; ++u) {
      const uint32_t t = t0 + u;
      if (t < D && (t == 0 || key[t] != key[t - 1])) ++loc;
    }
    const uint32_t inc = wave_incl_scan(loc);
    if (lane == kWave - 1) wsum[wid] = inc;
    __syncthreads();
    uint32_t run = inc - loc;
    for (int x = 0; x < wid; ++x) run += wsum[x];
#pragma unroll
    for (uint32_t u = 0; u < kPer; ++u) {
      const uint32_t t = t0 + u;
      if (t < D) {
        if (t == 0 || key[t] != key[t - 1]) ++run;
        rk[t] = run - 1;
      }
    }
  }
  __syncthreads();
  // per rank (at its first slot): size and liveness, summed over the slots
  // that share it (several degrees share a rank only when their values d * w
  // coincide: when w = 0 in F_p; in Z/2^64 when 2^64 divides (d - d') w,
  // which for degrees below 2^32 needs more than 32 trailing zero bits in w)
  {
    uint32_t cnt_loc = 0, live_loc = 0;
#pragma unroll
    for (uint32_t u = 0; u < kPer; ++u) {
      const uint32_t t = t0 + u;
      if (t < D && (t == 0 || rk[t] != rk[t - 1])) {
        uint32_t size = 0;
        bool nonnull = false;
        uint32_t s = t;
        for (; s < D && rk[s] == rk[t]; ++s) {
          size += d.dcount[deg[s]];
          nonnull = nonnull || deg[s] > 0;
        }
        d.rdeg[rk[t]] = s == t + 1 ? deg[t] : kDegMixed;
        const bool live = size >= 2 && nonnull;
        // stash size and liveness in the rank table entry of the first slot
        d.roff[rk[t]] = live ? size : 0u;
        cnt_loc += live ? size : 0u;
        live_loc += live ? 1u : 0u;
      }
    }
    __syncthreads();
    const uint32_t inc = wave_incl_scan(cnt_loc);
    const uint32_t inc2 = wave_incl_scan(live_loc);
    if (lane == kWave - 1) {
      wsum[wid] = inc;
      wsum2[wid] = inc2;
    }
    __syncthreads();
    uint32_t off = inc - cnt_loc, jn = inc2 - live_loc;
    uint32_t tot = 0, totj = 0;
    for (int x = 0; x < kDegThreads / kWave; ++x) {
      if (x < wid) {
        off += wsum[x];
        jn += wsum2[x];
      }
      tot += wsum[x];
      totj += wsum2[x];
    }
#pragma unroll
    for (uint32_t u = 0; u < kPer; ++u) {
      const uint32_t t = t0 + u;
      if (t < D && (t == 0 || rk[t] != rk[t - 1])) {
        const uint32_t r = rk[t];
        const uint32_t size = d.roff[r];
        const bool live = size != 0;
        d.rj[r] = live ? jn : 0xFFFFFFFFu;
        d.roff[r] = off;
        if (live) {
          ctx.lcold[jn] = r;
          ctx.loff[jn] = off;
          ctx.llen[jn] = size;
        }
        off += size;
        jn += live ? 1u : 0u;
      }
    }
    if (threadIdx.x == 0) {
      const uint32_t k_new = D ? rk[D - 1] + 1 : 0;
      st->n_live2 = totj;
      st->nl2 = tot;
      st->k_new = k_new;
      st->nosplit = k_new == st->k ? 1u : 0u;
      st->split_any = 1u - st->nosplit;
    }
  }
  __syncthreads();
  // degree table -> rank | flags
  for (uint32_t t = threadIdx.x; t < D; t += kDegThreads) {
    const uint32_t r = rk[t];
    d.dcount[deg[t]] = r | (d.rj[r] != 0xFFFFFFFFu ? kDegLive : 0u) |
                       (d.rdeg[r] == kDegMixed ? kDegShared : 0u);
  }
}

// Class index and row length of every member-list position.  Both are the
// same over a live class's range (the class of its rank, the rank's degree),
// so they are written here in position order, four positions per thread;
// k_deg_place writes the member's own row length only in a rank that several
// degrees share.  Runs before k_deg_place.
__global__ void __launch_bounds__(kBlock) k_deg_fill(Ctx ctx, DegScratch d) {
  const DevState* st = ctx.st;
  if (*d.nd > kDegRanks || st->nosplit) return;
  const uint32_t nl = st->nl2, J = st->n_live2;  // J <= kDegRanks
  __shared__ uint32_t off[kDegRanks];
  __shared__ uint32_t dg[kDegRanks];
  for (uint32_t j = threadIdx.x; j < J; j += kBlock) {
    off[j] = ctx.loff[j];
    dg[j] = d.rdeg[ctx.lcold[j]];
  }
  __syncthreads();
  const bool vec = (((uintptr_t)ctx.qcls | (uintptr_t)ctx.rl) & 15) == 0;
  const uint32_t stride = gridDim.x * kBlock * 4;
  for (uint32_t q0 = (blockIdx.x * kBlock + threadIdx.x) * 4; q0 < nl; q0 += stride) {
    // the class holding q0: last j with off[j] <= q0 (off[0] = 0, J >= 1)
    uint32_t lo = 0, hi = J - 1;
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) >> 1;
      if (off[mid] <= q0) lo = mid; else hi = mid - 1;
    }
    uint32_t qc[4], rl[4];
    uint32_t j = lo;
#pragma unroll
    for (uint32_t u = 0; u < 4; ++u) {
      while (j + 1 < J && off[j + 1] <= q0 + u) ++j;
      qc[u] = j;
      rl[u] = dg[j];
    }
    if (vec && q0 + 4 <= nl) {
      *(uint4*)(ctx.qcls + q0) = make_uint4(qc[0], qc[1], qc[2], qc[3]);
      *(uint4*)(ctx.rl + q0) = make_uint4(rl[0], rl[1], rl[2], rl[3]);
    } else {
      for (uint32_t u = 0; u < 4 && q0 + u < nl; ++u) {
        ctx.qcls[q0 + u] = qc[u];
        ctx.rl[q0 + u] = rl[u];
      }
    }
  }
}

// Placement of the nodes of the live classes, class after class, as a
// counting sort over blocks: every block counts its nodes per rank (a
// column of the rank x block matrix m), each rank's row is scanned into
// offsets from the rank's first position, and every block places its nodes
// from its own offsets.  No block contends with another for a cursor.
__device__ __forceinline__ void deg_block_range(uint32_t n, uint32_t* lo, uint32_t* hi) {
  const uint32_t per = ((n + gridDim.x - 1) / gridDim.x + kBlock - 1) / kBlock * kBlock;
  *lo = min(n, blockIdx.x * per);
  *hi = min(n, *lo + per);
}

template <bool RP64>
__global__ void __launch_bounds__(kBlock) k_deg_count(Ctx ctx, DegScratch d, uint32_t* m) {
  const DevState* st = ctx.st;
  if (*d.nd > kDegRanks || st->nosplit) return;
  __shared__ uint32_t lc[kDegRanks];
  const uint32_t K = st->k_new, nblk = gridDim.x;
  uint32_t lo, hi;
  deg_block_range(ctx.n, &lo, &hi);
  for (uint32_t r = threadIdx.x; r < K; r += kBlock) lc[r] = 0;
  __syncthreads();
  for (uint32_t i0 = lo + threadIdx.x; i0 < hi; i0 += kBlock * kDegStep) {
    uint32_t g[kDegStep], e[kDegStep];
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) {
      const uint32_t i = i0 + u * kBlock;
      g[u] = i < hi ? degree_of(ctx, i, RP64) : 0u;
    }
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) e[u] = i0 + u * kBlock < hi ? d.dcount[g[u]] : 0u;
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u)
      if (e[u] & kDegLive) atomicAdd(&lc[e[u] & kDegRankMask], 1u);
  }
  __syncthreads();
  for (uint32_t r = threadIdx.x; r < K; r += kBlock) m[(uint64_t)r * nblk + blockIdx.x] = lc[r];
}

// One block per rank: its row of m becomes the first member-list position
// of each block's nodes of that rank.
__global__ void __launch_bounds__(kBlock) k_deg_rowscan(Ctx ctx, DegScratch d, uint32_t* m,
                                                        uint32_t nblk) {
  const DevState* st = ctx.st;
  if (*d.nd > kDegRanks || st->nosplit) return;
  const uint32_t K = st->k_new;
  __shared__ uint32_t sh[kBlock / kWave];
  for (uint32_t r = blockIdx.x; r < K; r += gridDim.x) {
    uint32_t* row = m + (uint64_t)r * nblk;
    uint32_t carry = d.roff[r];
    for (uint32_t b0 = 0; b0 < nblk; b0 += kBlock) {
      const uint32_t b = b0 + threadIdx.x;
      const uint32_t v = b < nblk ? row[b] : 0u;
      uint32_t tot;
      const uint32_t ex = block_excl_scan(v, sh, &tot);
      if (b < nblk) row[b] = carry + ex;
      carry += tot;
    }
  }
}

// New colour of every node; members of live classes placed from their
// block's offsets.  Nothing of the live state is read in this round, so the
// lists are written in place.
template <bool RP64>
__global__ void __launch_bounds__(kBlock) k_deg_place(Ctx ctx, DegScratch d, const uint32_t* m) {
  const DevState* st = ctx.st;
  if (*d.nd > kDegRanks || st->nosplit) return;
  __shared__ uint32_t lc[kDegRanks];
  const uint32_t K = st->k_new, nblk = gridDim.x;
  uint32_t lo, hi;
  deg_block_range(ctx.n, &lo, &hi);
  for (uint32_t r = threadIdx.x; r < K; r += kBlock) lc[r] = m[(uint64_t)r * nblk + blockIdx.x];
  __syncthreads();
  const uint32_t lane = lane_id();
  // the loop bounds are the same for the whole wave (hi - lo is a multiple of
  // kBlock or the block's last range; lanes past hi take part inactive)
  for (uint32_t i0 = lo + threadIdx.x - lane; i0 < hi; i0 += kBlock * kDegStep) {
    uint64_t r0[kDegStep];
    uint32_t g[kDegStep], e[kDegStep];
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) {
      const uint32_t i = i0 + lane + u * kBlock;
      r0[u] = 0;
      g[u] = 0;
      if (i < hi) {
        r0[u] = RP64 ? ctx.rp64[i] : ctx.rp32[i];
        g[u] = (uint32_t)((RP64 ? ctx.rp64[i + 1] : (uint64_t)ctx.rp32[i + 1]) - r0[u]);
      }
    }
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) e[u] = i0 + lane + u * kBlock < hi ? d.dcount[g[u]] : 0u;
#pragma unroll
    for (uint32_t u = 0; u < kDegStep; ++u) {
      const uint32_t i = i0 + lane + u * kBlock;
      const bool in = i < hi;
      const uint32_t r = e[u] & kDegRankMask;
      if (in) ctx.c[i] = r;
      const bool live = in && (e[u] & kDegLive) != 0;
      // slots: one LDS atomic per rank present in the wave, ranks of the
      // lanes inside it by their position
      const unsigned long long peers = wave_peers(r, live);
      const int ldr = live ? __ffsll((long long)peers) - 1 : (int)lane;
      uint32_t b = 0;
      if (live && (int)lane == ldr) b = atomicAdd(&lc[r], (uint32_t)__popcll(peers));
      b = __shfl(b, ldr, kWave);
      if (in && !live && ctx.pos_deg) ctx.pos_deg[i] = 0xFFFFFFFFu;
      if (live) {
        const uint32_t q = b + (uint32_t)__popcll(peers & ((1ull << lane) - 1));
        if (ctx.pos_deg) ctx.pos_deg[i] = q;
        ctx.lperm[q] = i;
        ctx.rs[q] = r0[u];
        if (e[u] & kDegShared) ctx.rl[q] = g[u];  // k_deg_fill wrote the rest
      }
    }
  }
}

}  // namespace wl
