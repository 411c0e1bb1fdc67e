// Device kernels of Algorithm 2 (Section 4.2): local row pointers of a batch
// and the quotient graph of Definition "Quotient Graph" (Eq. sc).
//
// Quotient: row of block B = row of its representative (smallest node) with
// every column mapped to its block and the weights summed per target block.
// Per chunk of rows, every entry of a representative row becomes the key
// (B - B_first) << 30 | block(column) with its weight as payload; the keys
// are sorted with the relabel machinery (one segment, keys in 'keys'), equal
// keys are flagged and ranked by the scan, and the weights are reduced per
// rank.
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

// One wave per row of the chunk.  qoff[r] = position of row r's first key
// (only representative rows have keys).
__global__ void __launch_bounds__(kBlock) k_q_keys(Ctx ctx, const uint64_t* rp,
                                                   const uint32_t* col,
                                                   const uint32_t* wt,
                                                   const uint32_t* blk,
                                                   const uint8_t* isrep,
                                                   const uint64_t* qoff,
                                                   uint32_t nrows, uint32_t row0,
                                                   uint32_t bfirst) {
  const uint32_t lane = lane_id();
  const uint32_t nwaves = gridDim.x * (kBlock / kWave);
  for (uint32_t r = blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; r < nrows;
       r += nwaves) {
    const uint32_t g = row0 + r;
    if (!isrep[g]) continue;
    const uint64_t brel = (uint64_t)(blk[g] - bfirst);
    const uint64_t beg = rp[r], end = rp[r + 1], at = qoff[r];
    for (uint64_t e = beg + lane; e < end; e += kWave) {
      ctx.keys[at + (e - beg)] = (brel << kQShift) | blk[col[e]];
      ctx.perm[at + (e - beg)] = wt ? wt[e] : 1u;
    }
  }
}

// Before the sort: one segment [0, cnt) (k = 1), clear the reduce slots and
// the entry counts of the chunk's blocks.
__global__ void __launch_bounds__(kBlock) k_q_begin(Ctx ctx, uint32_t cnt, uint32_t* qdeg,
                                                    uint32_t nblocks) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctx.st->k = 1;
    ctx.st->done = 0;
    ctx.cstart[0] = 0;
    ctx.cstart[1] = cnt;
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
  for (uint32_t d = blockIdx.x * kBlock + threadIdx.x; d < nd; d += gridDim.x * kBlock) {
    const uint64_t key = ctx.z[d];
    const uint64_t w = qw[d];
    if (w > 0xFFFFFFFFull) atomicOr(&ctx.st->err, kErrQuotientWeight);
    qcol[d] = (uint32_t)(key & mask);
    qwt[d] = (uint32_t)w;
    atomicAdd(&qdeg[key >> kQShift], 1u);
  }
}

}  // namespace wl
