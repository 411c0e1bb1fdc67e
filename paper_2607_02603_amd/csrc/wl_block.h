// Workgroup-level scan primitives for 256-thread (4 x wave64) blocks.
#pragma once
#include "wl_ctx.h"
#include "wl_device.h"

namespace wl {

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    uint32_t o = __shfl_up(v, off, kWave);
    if (lane >= off) v += o;
  }
  return v;
}

// Exclusive scan over the 256 threads of a block; returns the thread's
// exclusive prefix and writes the block total to *total.  'sh' must hold
// kBlock / kWave words of shared memory.  Contains __syncthreads().
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* sh,
                                                    uint32_t* total) {
  const int lane = lane_id();
  const int wid = threadIdx.x / kWave;
  uint32_t inc = wave_incl_scan(v);
  if (lane == kWave - 1) sh[wid] = inc;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kBlock / kWave; ++w) {
    uint32_t s = sh[w];
    if (w < wid) base += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

// Exclusive scan in place of p[0, n), n <= 4 * kBlock, by one block: each
// thread takes four consecutive items, so one block scan does it.  Returns
// the total.  Contains __syncthreads().
__device__ __forceinline__ uint32_t block_scan_small(uint32_t* p, uint32_t n, uint32_t* sh) {
  const uint32_t i0 = 4 * threadIdx.x;
  uint32_t v[4], s = 0;
#pragma unroll
  for (uint32_t u = 0; u < 4; ++u) {
    v[u] = i0 + u < n ? p[i0 + u] : 0u;
    s += v[u];
  }
  uint32_t tot;
  uint32_t run = block_excl_scan(s, sh, &tot);
#pragma unroll
  for (uint32_t u = 0; u < 4; ++u)
    if (i0 + u < n) {
      p[i0 + u] = run;
      run += v[u];
    }
  return tot;
}

// Sum of p[0, b) and, in *total, of p[0, n), by every thread of the block
// (n <= 4 * kBlock: block sums of a device-wide scan, each block of the
// scan's last launch taking its own offset instead of a separate launch
// scanning them).  Contains __syncthreads().
__device__ __forceinline__ uint32_t block_part_prefix(const uint32_t* p, uint32_t n,
                                                      uint32_t b, uint32_t* sh,
                                                      uint32_t* total) {
  uint32_t below = 0, all = 0;
  for (uint32_t i = threadIdx.x; i < n; i += kBlock) {
    const uint32_t v = p[i];
    all += v;
    below += i < b ? v : 0u;
  }
  uint32_t tb, ta;
  block_excl_scan(below, sh, &tb);
  block_excl_scan(all, sh, &ta);
  *total = ta;
  return tb;
}

// Chained scan (decoupled look-back) over chunks handed out in ticket order:
// chunk c publishes its total, then its inclusive prefix, in desc[c]; chunk
// c + 1 adds totals walking back until it finds an inclusive prefix.  A
// descriptor packs an epoch (bits 63..34: the round and the scan site, so
// words left by an earlier scan read as not ready), a state (bits 33..32:
// 1 total, 2 inclusive prefix) and the 32-bit value, so relaxed agent-scope
// atomics carry everything a reader needs and no fence is issued.  Chunks
// are taken by ticket (an atomic counter), so every chunk a block waits for
// belongs to a block that is already running: the walk ends.  A wait longer
// than max_spins polls (by default kChainSpins, far beyond any real wait)
// gives up, so a kernel never hangs: it sets kErrChain and stops the device
// (kStoppedOnError), so that no later kernel uses the unfinished result.
constexpr uint32_t kErrChain = 64u;       // DevState::err bit
constexpr uint32_t kStoppedOnError = 5;   // DevState::done: stopped, err says why
constexpr uint32_t kChainSpins = 1u << 22;
constexpr int kChainSplits = 0, kChainFlags = 1, kChainA = 2, kChainB = 3;  // sites

__device__ __forceinline__ uint32_t chain_epoch(uint32_t round, int site) {
  return (round * 4u + (uint32_t)site) & 0x3FFFFFFFu;
}

// Every thread of the block calls it with the same c and total; returns the
// exclusive prefix of chunk c.  The first wave walks back kWave descriptors
// per poll (lane l reads chunk p - l).  Contains __syncthreads().
__device__ __forceinline__ uint32_t chain_prefix(unsigned long long* desc, uint32_t c,
                                                 uint32_t total, uint32_t epoch,
                                                 uint32_t max_spins, DevState* st,
                                                 uint32_t* sh1) {
  if (threadIdx.x < kWave) {
    const int lane = (int)threadIdx.x;
    const unsigned long long tag = (unsigned long long)epoch << 34;
    uint32_t excl = 0;
    if (c > 0) {
      if (lane == 0)
        __hip_atomic_store(&desc[c], tag | (1ull << 32) | total, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      int64_t p = (int64_t)c - 1;
      uint32_t spins = 0;
      while (true) {
        const int64_t idx = p - lane;
        // before chunk 0: an inclusive prefix of 0 (chunk 0 itself only ever
        // publishes its inclusive prefix, so the walk stops there first)
        uint32_t state = 2, val = 0;
        if (idx >= 0) {
          const unsigned long long d =
              __hip_atomic_load(&desc[idx], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          state = (uint32_t)(d >> 34) == epoch ? (uint32_t)(d >> 32) & 3u : 0u;
          val = (uint32_t)d;
        }
        const unsigned long long inc = __ballot(state == 2);
        const unsigned long long wait = __ballot(state == 0);
        // lanes up to the nearest inclusive prefix (all lanes if none) must be ready
        const int first = inc ? __ffsll((long long)inc) - 1 : kWave;
        const unsigned long long need = first >= kWave - 1 ? ~0ull : (2ull << first) - 1;
        if (wait & need) {
          if (++spins > max_spins) {
            if (lane == 0) {
              atomicOr(&st->err, kErrChain);
              st->done = kStoppedOnError;
            }
            break;
          }
          __builtin_amdgcn_s_sleep(1);
          continue;
        }
        uint32_t v = lane <= first ? val : 0u;
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
        excl += v;
        if (first < kWave) break;
        p -= kWave;
      }
    }
    if (lane == 0) {
      __hip_atomic_store(&desc[c], tag | (2ull << 32) | (excl + total), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      *sh1 = excl;
    }
  }
  __syncthreads();
  const uint32_t r = *sh1;
  __syncthreads();
  return r;
}

// Next chunk ticket of a chained scan for the whole block.  Contains
// __syncthreads().
__device__ __forceinline__ uint32_t chain_ticket(uint32_t* counter, uint32_t* sh1) {
  if (threadIdx.x == 0) *sh1 = atomicAdd(counter, 1u);
  __syncthreads();
  const uint32_t t = *sh1;
  __syncthreads();
  return t;
}

// Appends 'want' items to a device list: one atomic per block, slots
// handed out by a block scan (order inside the list is irrelevant).
// Contains __syncthreads(); every thread of the block must call it.
__device__ __forceinline__ uint32_t block_append(bool want, uint32_t* counter,
                                                 uint32_t* sh, uint32_t* base_sh) {
  uint32_t tot;
  const uint32_t ex = block_excl_scan(want ? 1u : 0u, sh, &tot);
  if (threadIdx.x == 0) *base_sh = tot ? atomicAdd(counter, tot) : 0u;
  __syncthreads();
  const uint32_t at = *base_sh + ex;
  __syncthreads();
  return at;
}

// Appends items of four kinds to four device lists at once: 'kind' in
// [0, 4), or 4 and above for no item; returns the item's slot in its kind's
// list (order inside a list is irrelevant).  Ranks inside a wave come from
// ballots, one atomic per kind and block, the four issued together.
// Contains __syncthreads(); every thread of the block must call it.
__device__ __forceinline__ uint32_t block_append4(uint32_t kind, uint32_t* c0, uint32_t* c1,
                                                  uint32_t* c2, uint32_t* c3) {
  __shared__ uint32_t wc[kBlock / kWave][4];
  __shared__ uint32_t base4[4];
  const int lane = lane_id(), wid = threadIdx.x / kWave;
  uint32_t rank = 0;
#pragma unroll
  for (uint32_t k = 0; k < 4; ++k) {
    const unsigned long long m = __ballot(kind == k);
    if (kind == k) rank = (uint32_t)__popcll(m & ((1ull << lane) - 1));
    if (lane == 0) wc[wid][k] = (uint32_t)__popcll(m);
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    const uint32_t k = threadIdx.x;
    uint32_t tot = 0;
    for (int w = 0; w < kBlock / kWave; ++w) {
      const uint32_t c = wc[w][k];
      wc[w][k] = tot;
      tot += c;
    }
    uint32_t* const ctr = k == 0 ? c0 : (k == 1 ? c1 : (k == 2 ? c2 : c3));
    base4[k] = tot ? atomicAdd(ctr, tot) : 0u;
  }
  __syncthreads();
  const uint32_t at = kind < 4 ? base4[kind] + wc[wid][kind] + rank : 0u;
  __syncthreads();
  return at;
}

// Lane l's value of v, for a lane index l that is the same in the whole
// wave (a register read, not an LDS permute as a shuffle is).
__device__ __forceinline__ uint64_t read_lane64(uint64_t v, int l) {
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(v >> 32), l) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
}

// Lanes of the wave that are active and hold the same key as this lane
// (0 for an inactive lane); one pass per distinct key among the active
// lanes.  Every lane of the calling control flow must call it.
__device__ __forceinline__ unsigned long long wave_peers(uint32_t key, bool active) {
  unsigned long long todo = __ballot(active);
  unsigned long long mine = 0;
  while (todo) {
    const int leader = __ffsll((long long)todo) - 1;
    const uint32_t lk = (uint32_t)__builtin_amdgcn_readlane((int)key, leader);
    const bool same = active && key == lk;
    const unsigned long long m = __ballot(same);
    if (same) mine = m;
    todo &= ~m;
  }
  return mine;
}

}  // namespace wl
