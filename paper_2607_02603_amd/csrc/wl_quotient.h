// Device kernels of Algorithm 2 (Section 4.2): local row pointers of a batch
// and the quotient graph of Definition "Quotient Graph" (Eq. sc).
//
// Quotient: row of block B = row of its representative (smallest node) with
// every column mapped to its block and the weights summed per target block.
// Per chunk of rows, every entry of a representative row becomes the key
// (B - B_first) << 30 | block(column) with its weight as payload; the keys
// are sorted with the relabel machinery (keys in 'keys'), one segment per
// row, so that most rows are sorted by one wave, equal keys are flagged and
// ranked by the scan, and the weights are reduced per rank.
#pragma once
#include "wl_relabel.h"

namespace wl {

constexpr int kQShift = 30;  // bits of the target block in a quotient key

// rp_out[i] = rp_in[i] - rp_in[0] for i <= nrows (input uint32 or uint64).
template <typename T>
__global__ void __launch_bounds__(kBlock) k_rebase_rows(const T* rp_in, uint64_t* rp_out,
                                                        uint32_t nrows) {
  const uint64_t base = rp_in[0];
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i <= nrows;
       i += gridDim.x * kBlock)
    rp_out[i] = (uint64_t)rp_in[i] - base;
}

// Keys of the chunk's representative rows.  qoff[r] = position of row r's
// first key (only representative rows have keys).  One entry per lane, so
// that the column indices are read and the keys written in runs: a wave
// finds the rows of its 64 consecutive entries among the 64 rows that
// follow the row of its first entry (a binary search), and the few lanes
// whose entry lies beyond them (empty rows in between) search on their own.
__device__ __forceinline__ uint32_t q_row_of(const uint64_t* rp, uint32_t nrows, uint64_t e) {
  uint32_t lo = 0, hi = nrows - 1;  // last r with rp[r] <= e
  while (lo < hi) {
    const uint32_t mid = (lo + hi + 1) >> 1;
    if (rp[mid] <= e) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ void __launch_bounds__(kBlock) k_q_keys(Ctx ctx, const uint64_t* rp,
                                                   const uint32_t* col,
                                                   const uint32_t* wt,
                                                   const uint32_t* blk,
                                                   const uint8_t* isrep,
                                                   const uint64_t* qoff,
                                                   uint32_t nrows, uint32_t row0,
                                                   uint32_t bfirst) {
  const uint32_t lane = lane_id();
  const uint64_t ent = rp[nrows];
  // 'base' is the same for all lanes of a wave (the shuffles need them all)
  for (uint64_t base = blockIdx.x * (uint64_t)kBlock + threadIdx.x - lane; base < ent;
       base += (uint64_t)gridDim.x * kBlock) {
    const uint64_t e = base + lane;
    const uint32_t r0 =
        (uint32_t)__builtin_amdgcn_readlane((int)(lane == 0 ? q_row_of(rp, nrows, base) : 0u), 0);
    // window: row starts rp[r0 + 1 .. r0 + 64]; lane j holds rp[r0 + 1 + j]
    const uint32_t rj = r0 + 1 + lane;
    const uint64_t sj = rj <= nrows ? rp[rj] : ~0ull;
    // row of e = r0 + (number of window starts <= e), counted by every lane
    // of the wave; an entry past the window searches on its own
    uint32_t cnt = 0;
#pragma unroll 8
    for (int j = 0; j < kWave; ++j) cnt += read_lane64(sj, j) <= e ? 1u : 0u;
    if (e >= ent) continue;
    const uint32_t r = cnt == (uint32_t)kWave ? q_row_of(rp, nrows, e) : r0 + cnt;
    if (!isrep[row0 + r]) continue;
    const uint64_t brel = (uint64_t)(blk[row0 + r] - bfirst);
    const uint64_t at = qoff[r] + (e - rp[r]);
    ctx.keys[at] = (brel << kQShift) | blk[col[e]];
    ctx.perm[at] = wt ? wt[e] : 1u;
  }
}

// Before the sort: the segments (nseg > 0: one per non-empty row, whose
// starts the host has put in cstart; 0: one segment [0, cnt)), clear the
// reduce slots and the entry counts of the chunk's blocks.
__global__ void __launch_bounds__(kBlock) k_q_begin(Ctx ctx, uint32_t cnt, uint32_t* qdeg,
                                                    uint32_t nblocks, uint32_t nseg) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctx.st->k = nseg ? nseg : 1;
    ctx.st->done = 0;
    if (!nseg) {
      ctx.cstart[0] = 0;
      ctx.cstart[1] = cnt;
    }
  }
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < cnt; i += gridDim.x * kBlock)
    ctx.x[i] = 0;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < nblocks; i += gridDim.x * kBlock)
    qdeg[i] = 0;
}

// After the sort and the scan: distinct keys and their summed weights.
__global__ void __launch_bounds__(kBlock) k_q_reduce(Ctx ctx, uint32_t cnt) {
  unsigned long long* qw = (unsigned long long*)ctx.x;
  for (uint32_t p = blockIdx.x * kBlock + threadIdx.x; p < cnt; p += gridDim.x * kBlock) {
    const uint32_t id = ctx.ids[p];
    atomicAdd(&qw[id], (unsigned long long)ctx.perm[p]);
    if (ctx.flags[p]) ctx.z[id] = ctx.keys[p];
  }
}

constexpr uint32_t kErrQuotientWeight = 8u;  // DevState::err bit

// The distinct entries in key order (block, then target) as column and weight
// arrays, and the number of entries of every block.  Weights are reduced to
// 32 bits; a larger sum sets an error bit.
__global__ void __launch_bounds__(kBlock) k_q_emit(Ctx ctx, uint32_t cnt, uint32_t* qcol,
                                                   uint32_t* qwt, uint32_t* qdeg) {
  const uint32_t nd = min(ctx.st->k_new, cnt);
  const unsigned long long* qw = (const unsigned long long*)ctx.x;
  const uint64_t mask = (1ull << kQShift) - 1;
  const uint32_t lane = lane_id();
  for (uint32_t d = blockIdx.x * kBlock + threadIdx.x; d < nd; d += gridDim.x * kBlock) {
    const uint64_t key = ctx.z[d];
    const uint64_t w = qw[d];
    if (w > 0xFFFFFFFFull) atomicOr(&ctx.st->err, kErrQuotientWeight);
    qcol[d] = (uint32_t)(key & mask);
    qwt[d] = (uint32_t)w;
    // the entries are in block order: the lanes of one block add their count
    // with one atomic
    const uint32_t b = (uint32_t)(key >> kQShift);
    const unsigned long long peers = wave_peers(b, true);
    if ((int)lane == __ffsll((long long)peers) - 1) atomicAdd(&qdeg[b], (uint32_t)__popcll(peers));
  }
}

}  // namespace wl
