// Exact stability certificate (Definition "Stable Coloring"): a colouring is
// stable when every two nodes of one colour class have the same total
// out-weight into every class.  Deterministic: no random values are drawn.
//
// Every row that matters (a row of a class with two or more nodes) becomes
// its sorted list of neighbour colours, kept in CSR layout in 'keys'; for
// weighted graphs the entry weight rides in the low 32 bits of a 64-bit key.
// Each node is then compared with the smallest node of its class:
//   unweighted  the sorted colour lists must be equal (equal multisets);
//   weighted    the lists of (colour, summed weight) runs must be equal,
//               runs whose weights sum to zero being absent (an entry of
//               weight 0 adds nothing to a_{i,B}).
// Row sorts:
//   <= 64 entries         bitonic network across the lanes of one wave;
//   <= kVChunk entries    bitonic network in LDS, one workgroup per row;
//   longer rows           every aligned chunk of kVChunk entries is sorted in
//                         LDS, then the chunks are merged in place by the
//                         remaining steps of a bitonic network in which every
//                         comparator puts the smaller key first (the first
//                         step of each merge compares a position with its
//                         mirror in the block).  Positions past the end of the
//                         row act as +infinity, so nothing is padded in memory:
//                         a comparator whose upper position is past the end
//                         never moves anything.
#pragma once
#include "wl_block.h"

namespace wl {

constexpr uint32_t kVChunk = 4096;
constexpr uint32_t kVErrColor = 1u;     // a colour >= k
constexpr uint32_t kVErrMismatch = 2u;  // two nodes of one class differ

struct VerState {
  uint32_t err;
  uint32_t n_mid;         // rows of 65 .. kVChunk entries to sort
  uint32_t n_hub;         // rows longer than kVChunk
  uint32_t n_hub_chunks;  // kVChunk-sized chunks over all hub rows
  uint64_t max_pow;       // largest padded (power of two) hub row length
};

template <typename K>
struct VerCtx {
  uint32_t n, k;
  const uint32_t* rp32;
  const uint64_t* rp64;
  const uint32_t* col;
  const uint32_t* wgt;
  const uint32_t* color;
  VerState* st;
  uint32_t* rep;        // k: smallest node of each class
  uint8_t* multi;       // k: 1 if the class has two or more nodes
  uint32_t* mid;        // rows to sort in LDS
  uint32_t* hub;        // rows longer than kVChunk
  uint32_t* hub_off;    // n_hub + 1: exclusive scan of chunks per hub row
  K* keys;              // nnz: sorted neighbour colours, CSR layout
};

template <typename K>
__device__ __forceinline__ uint64_t v_beg(const VerCtx<K>& v, uint32_t i) {
  return v.rp64 ? v.rp64[i] : (uint64_t)v.rp32[i];
}

template <typename K>
__device__ __forceinline__ K v_inf();
template <>
__device__ __forceinline__ uint32_t v_inf<uint32_t>() { return 0xFFFFFFFFu; }
template <>
__device__ __forceinline__ uint64_t v_inf<uint64_t>() { return ~0ull; }

// Key of entry e: colour of its column (high 32 bits when weighted, with the
// weight below).  Colours are < k <= 2^32 - 1, so every key is below v_inf.
template <typename K>
__device__ __forceinline__ K v_key(const VerCtx<K>& v, uint64_t e);
template <>
__device__ __forceinline__ uint32_t v_key<uint32_t>(const VerCtx<uint32_t>& v, uint64_t e) {
  return v.color[v.col[e]];
}
template <>
__device__ __forceinline__ uint64_t v_key<uint64_t>(const VerCtx<uint64_t>& v, uint64_t e) {
  return ((uint64_t)v.color[v.col[e]] << 32) | v.wgt[e];
}

template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_clear(VerCtx<K> v) {
  for (uint32_t b = blockIdx.x * kBlock + threadIdx.x; b < v.k; b += gridDim.x * kBlock) {
    v.rep[b] = 0xFFFFFFFFu;
    v.multi[b] = 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    v.st->err = 0;
    v.st->n_mid = 0;
    v.st->n_hub = 0;
    v.st->n_hub_chunks = 0;
    v.st->max_pow = 0;
  }
}

// Representative of every class: its smallest node.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_rep(VerCtx<K> v) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < v.n; i += gridDim.x * kBlock) {
    const uint32_t c = v.color[i];
    if (c >= v.k) {
      atomicOr(&v.st->err, kVErrColor);
      continue;
    }
    if (__hip_atomic_load(&v.rep[c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) > i)
      atomicMin(&v.rep[c], i);
  }
}

template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_multi(VerCtx<K> v) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < v.n; i += gridDim.x * kBlock) {
    const uint32_t c = v.color[i];
    if (v.rep[c] != i) v.multi[c] = 1;
  }
}

// Rows longer than one wave go to the LDS list or the hub list.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_bin(VerCtx<K> v) {
  __shared__ uint32_t sh[kBlock / kWave];
  __shared__ uint32_t base_sh;
  for (uint32_t i0 = blockIdx.x * kBlock; i0 < v.n; i0 += gridDim.x * kBlock) {
    const uint32_t i = i0 + threadIdx.x;
    uint64_t len = 0;
    if (i < v.n && v.multi[v.color[i]]) len = v_beg(v, i + 1) - v_beg(v, i);
    const bool mid = len > (uint64_t)kWave && len <= kVChunk;
    const bool hub = len > kVChunk;
    uint32_t tot;
    uint32_t ex = block_excl_scan(mid ? 1u : 0u, sh, &tot);
    if (threadIdx.x == 0) base_sh = tot ? atomicAdd(&v.st->n_mid, tot) : 0u;
    __syncthreads();
    if (mid) v.mid[base_sh + ex] = i;
    __syncthreads();
    ex = block_excl_scan(hub ? 1u : 0u, sh, &tot);
    if (threadIdx.x == 0) base_sh = tot ? atomicAdd(&v.st->n_hub, tot) : 0u;
    __syncthreads();
    if (hub) v.hub[base_sh + ex] = i;
    __syncthreads();
  }
}

// One wave per row of 1 .. 64 entries: keys, bitonic sort across lanes.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_sort_wave(VerCtx<K> v) {
  const uint32_t lane = lane_id();
  const uint32_t nwaves = gridDim.x * (kBlock / kWave);
  for (uint32_t i = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; i < v.n;
       i += nwaves) {
    if (!v.multi[v.color[i]]) continue;
    const uint64_t b = v_beg(v, i), len = v_beg(v, i + 1) - b;
    if (len == 0 || len > (uint64_t)kWave) continue;
    K key = lane < len ? v_key(v, b + lane) : v_inf<K>();
#pragma unroll
    for (uint32_t kk = 2; kk <= (uint32_t)kWave; kk <<= 1) {
#pragma unroll
      for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
        const K pk = __shfl_xor(key, (int)j, kWave);
        const bool up = (lane & kk) == 0;
        const bool lower = (lane & j) == 0;
        if ((lower == up) ? (pk < key) : (pk > key)) key = pk;
      }
    }
    if (lane < len) v.keys[b + lane] = key;
  }
}

// Ascending bitonic sort of s[0 .. P) in LDS (P a power of two, P >= 2).
// Contains __syncthreads(); every thread of the block must call it.
template <typename K>
__device__ __forceinline__ void lds_bitonic(K* s, uint32_t P) {
  for (uint32_t kk = 2; kk <= P; kk <<= 1) {
    for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < P; i += kBlock) {
        const uint32_t l = i ^ j;
        if (l > i) {
          const bool asc = (i & kk) == 0;
          const K a = s[i], c = s[l];
          if ((a > c) == asc) {
            s[i] = c;
            s[l] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

// One workgroup per row of 65 .. kVChunk entries.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_sort_mid(VerCtx<K> v) {
  __shared__ K s[kVChunk];
  const uint32_t nm = v.st->n_mid;
  for (uint32_t q = blockIdx.x; q < nm; q += gridDim.x) {
    const uint32_t i = v.mid[q];
    const uint64_t b = v_beg(v, i);
    const uint32_t len = (uint32_t)(v_beg(v, i + 1) - b);
    uint32_t P = 2;
    while (P < len) P <<= 1;
    for (uint32_t t = threadIdx.x; t < P; t += kBlock)
      s[t] = t < len ? v_key(v, b + t) : v_inf<K>();
    __syncthreads();
    lds_bitonic(s, P);
    for (uint32_t t = threadIdx.x; t < len; t += kBlock) v.keys[b + t] = s[t];
    __syncthreads();
  }
}

// One block: chunks per hub row (exclusive scan) and the largest padded
// length, which sets the merge stages the host launches.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_hub_plan(VerCtx<K> v) {
  __shared__ uint32_t sh[kBlock / kWave];
  __shared__ unsigned long long mx;
  if (threadIdx.x == 0) mx = 0;
  __syncthreads();
  const uint32_t nh = v.st->n_hub;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nh; base += kBlock) {
    const uint32_t h = base + threadIdx.x;
    uint32_t nc = 0;
    if (h < nh) {
      const uint32_t i = v.hub[h];
      const uint64_t len = v_beg(v, i + 1) - v_beg(v, i);
      nc = (uint32_t)((len + kVChunk - 1) / kVChunk);
      uint64_t P = kVChunk;
      while (P < len) P <<= 1;
      atomicMax(&mx, (unsigned long long)P);
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan(nc, sh, &tot);
    if (h < nh) v.hub_off[h] = carry + ex;
    carry += tot;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    v.hub_off[nh] = carry;
    v.st->n_hub_chunks = carry;
    v.st->max_pow = mx;
  }
}

struct HubChunk {
  uint64_t base;  // first entry of the row
  uint64_t len;   // entries of the row
  uint64_t pos;   // position of the chunk's first entry inside the row
};

template <typename K>
__device__ __forceinline__ HubChunk hub_chunk(const VerCtx<K>& v, uint32_t t) {
  uint32_t lo = 0, hi = v.st->n_hub - 1;  // last h with hub_off[h] <= t
  while (lo < hi) {
    const uint32_t mid = (lo + hi + 1) >> 1;
    if (v.hub_off[mid] <= t) lo = mid; else hi = mid - 1;
  }
  const uint32_t i = v.hub[lo];
  HubChunk c;
  c.base = v_beg(v, i);
  c.len = v_beg(v, i + 1) - c.base;
  c.pos = (uint64_t)(t - v.hub_off[lo]) * kVChunk;
  return c;
}

__device__ __forceinline__ uint64_t pow2_at_least(uint64_t len) {
  uint64_t P = kVChunk;
  while (P < len) P <<= 1;
  return P;
}

// Stages of block size <= kVChunk: every aligned chunk of a hub row sorted.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_hub_sort_chunks(VerCtx<K> v) {
  __shared__ K s[kVChunk];
  const uint32_t nc = v.st->n_hub_chunks;
  for (uint32_t t = blockIdx.x; t < nc; t += gridDim.x) {
    const HubChunk c = hub_chunk(v, t);
    const uint64_t valid = min((uint64_t)kVChunk, c.len - c.pos);
    for (uint32_t q = threadIdx.x; q < kVChunk; q += kBlock)
      s[q] = q < valid ? v_key(v, c.base + c.pos + q) : v_inf<K>();
    __syncthreads();
    lds_bitonic(s, kVChunk);
    for (uint32_t q = threadIdx.x; q < valid; q += kBlock) v.keys[c.base + c.pos + q] = s[q];
    __syncthreads();
  }
}

template <typename K>
__device__ __forceinline__ void cmpx(K* a, K* b) {
  const K x = *a, y = *b;
  if (y < x) {
    *a = y;
    *b = x;
  }
}

// One global step of the merge of block size kk (kk > kVChunk) over every
// hub row: flip == 1 compares position i with its mirror i ^ (kk - 1) in the
// block, otherwise i with i + j (bit j of i clear; j >= kVChunk).  A chunk
// takes part when it holds lower positions of the step.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_hub_step(VerCtx<K> v, uint64_t kk, uint64_t j,
                                                       int flip) {
  const uint32_t nc = v.st->n_hub_chunks;
  for (uint32_t t = blockIdx.x; t < nc; t += gridDim.x) {
    const HubChunk c = hub_chunk(v, t);
    if (pow2_at_least(c.len) < kk) continue;
    const uint64_t bit = flip ? kk >> 1 : j;
    if (c.pos & bit) continue;
    K* row = v.keys + c.base;
    for (uint32_t q = threadIdx.x; q < kVChunk; q += kBlock) {
      const uint64_t i = c.pos + q;
      const uint64_t l = flip ? (i ^ (kk - 1)) : (i + j);
      if (l < c.len) cmpx(row + i, row + l);
    }
  }
}

// The steps j = kVChunk/2 .. 1 of the merge of block size kk, inside each
// chunk, in LDS.
template <typename K>
__global__ void __launch_bounds__(kBlock) k_v_hub_finish(VerCtx<K> v, uint64_t kk) {
  __shared__ K s[kVChunk];
  const uint32_t nc = v.st->n_hub_chunks;
  for (uint32_t t = blockIdx.x; t < nc; t += gridDim.x) {
    const HubChunk c = hub_chunk(v, t);
    if (pow2_at_least(c.len) < kk) continue;
    const uint64_t valid = min((uint64_t)kVChunk, c.len - c.pos);
    K* row = v.keys + c.base + c.pos;
    for (uint32_t q = threadIdx.x; q < kVChunk; q += kBlock)
      s[q] = q < valid ? row[q] : v_inf<K>();
    __syncthreads();
    for (uint32_t j = kVChunk >> 1; j > 0; j >>= 1) {
      for (uint32_t q = threadIdx.x; q < kVChunk; q += kBlock)
        if ((q & j) == 0) cmpx(s + q, s + (q | j));
      __syncthreads();
    }
    for (uint32_t q = threadIdx.x; q < valid; q += kBlock) row[q] = s[q];
    __syncthreads();
  }
}

// Unweighted: 16 lanes per node compare its sorted list with its
// representative's.
__global__ void __launch_bounds__(kBlock) k_v_compare(VerCtx<uint32_t> v) {
  constexpr uint32_t G = 16;
  const uint32_t sub = threadIdx.x % G;
  const uint32_t ngroups = gridDim.x * (kBlock / G);
  for (uint32_t i = blockIdx.x * (kBlock / G) + threadIdx.x / G; i < v.n; i += ngroups) {
    const uint32_t c = v.color[i];
    const uint32_t r = v.rep[c];
    if (r == i) continue;
    const uint64_t bi = v_beg(v, i), li = v_beg(v, i + 1) - bi;
    const uint64_t br = v_beg(v, r), lr = v_beg(v, r + 1) - br;
    bool bad = li != lr;
    if (!bad)
      for (uint64_t t = sub; t < li; t += G)
        if (v.keys[bi + t] != v.keys[br + t]) bad = true;
    if (bad) atomicOr(&v.st->err, kVErrMismatch);
  }
}

// Next run of equal colours with a nonzero weight sum at or after *p (end e);
// returns false when none is left.
__device__ __forceinline__ bool next_run(const uint64_t* keys, uint64_t* p, uint64_t e,
                                         uint32_t* color, uint64_t* sum) {
  while (*p < e) {
    const uint32_t c = (uint32_t)(keys[*p] >> 32);
    uint64_t s = 0;
    while (*p < e && (uint32_t)(keys[*p] >> 32) == c) s += keys[(*p)++] & 0xFFFFFFFFull;
    if (s) {
      *color = c;
      *sum = s;
      return true;
    }
  }
  return false;
}

// Weighted: one thread per node walks the (colour, weight sum) runs of its
// list and of its representative's in step.
__global__ void __launch_bounds__(kBlock) k_v_compare_w(VerCtx<uint64_t> v) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < v.n; i += gridDim.x * kBlock) {
    const uint32_t c = v.color[i];
    const uint32_t r = v.rep[c];
    if (r == i) continue;
    uint64_t pi = v_beg(v, i), ei = v_beg(v, i + 1);
    uint64_t pr = v_beg(v, r), er = v_beg(v, r + 1);
    for (;;) {
      uint32_t ci = 0, cr = 0;
      uint64_t si = 0, sr = 0;
      const bool hi = next_run(v.keys, &pi, ei, &ci, &si);
      const bool hr = next_run(v.keys, &pr, er, &cr, &sr);
      if (hi != hr || (hi && (ci != cr || si != sr))) {
        atomicOr(&v.st->err, kVErrMismatch);
        break;
      }
      if (!hi) break;
    }
  }
}

}  // namespace wl
