// GPU build of the seeded graph samplers (gen_common.h) for the large
// configurations.  Directed entry keys (u << 32 | v) of the symmetrised
// samples are bucketed by the high bits of the source so that each bucket
// can be sorted and deduplicated on its own; a count pass sizes the buckets
// and a scatter pass fills them (order inside a bucket is irrelevant: the
// caller sorts it).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gen_common.h"

namespace {

constexpr int kB = 256;
constexpr int kMaxBuckets = 1024;

struct Src {
  int kind;  // 0 = R-MAT, 1 = Chung-Lu
  uint32_t scale, ta, tab, tabc, n;
  uint64_t state;
  gen_perm perm;
  const uint64_t* thr;
  const uint32_t* alias;
};

__device__ __forceinline__ bool draw(const Src& S, uint64_t s, uint64_t* u,
                                     uint64_t* v) {
  if (S.kind == 0) {
    gen_rmat_raw(S.state, s, S.scale, S.ta, S.tab, S.tabc, u, v);
    *u = gen_apply_perm(&S.perm, *u);
    *v = gen_apply_perm(&S.perm, *v);
  } else {
    *u = gen_alias_draw(gen_u64(S.state, 2 * s), S.n, S.thr, S.alias);
    *v = gen_alias_draw(gen_u64(S.state, 2 * s + 1), S.n, S.thr, S.alias);
  }
  return *u != *v;
}

__global__ void __launch_bounds__(kB) k_count(Src S, uint64_t s0, uint64_t cnt,
                                              uint32_t shift, uint32_t nbk,
                                              unsigned long long* counts) {
  __shared__ uint32_t h[kMaxBuckets];
  for (uint32_t b = threadIdx.x; b < nbk; b += kB) h[b] = 0;
  __syncthreads();
  for (uint64_t q = blockIdx.x * (uint64_t)kB + threadIdx.x; q < cnt;
       q += (uint64_t)gridDim.x * kB) {
    uint64_t u, v;
    if (draw(S, s0 + q, &u, &v)) {
      atomicAdd(&h[u >> shift], 1u);
      atomicAdd(&h[v >> shift], 1u);
    }
  }
  __syncthreads();
  for (uint32_t b = threadIdx.x; b < nbk; b += kB)
    if (h[b]) atomicAdd(&counts[b], (unsigned long long)h[b]);
}

// Each block takes kPer samples per thread, ranks its keys per bucket in LDS
// and reserves room with one global atomic per bucket.
constexpr int kPer = 8;

__global__ void __launch_bounds__(kB) k_scatter(Src S, uint64_t s0, uint64_t cnt,
                                                uint32_t shift, uint32_t nbk,
                                                uint32_t blo, uint32_t bhi,
                                                unsigned long long* cursor,
                                                uint64_t* keys) {
  __shared__ uint32_t lcnt[kMaxBuckets];
  __shared__ unsigned long long lbase[kMaxBuckets];
  const uint64_t per_block = (uint64_t)kB * kPer;
  for (uint64_t base = blockIdx.x * per_block; base < cnt;
       base += (uint64_t)gridDim.x * per_block) {
    for (uint32_t b = threadIdx.x; b < nbk; b += kB) lcnt[b] = 0;
    __syncthreads();
    uint64_t key[2 * kPer];
    uint32_t slot[2 * kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const uint64_t q = base + (uint64_t)i * kB + threadIdx.x;
      uint64_t u = 0, v = 0;
      bool ok = q < cnt && draw(S, s0 + q, &u, &v);
      const bool oku = ok && (u >> shift) >= blo && (u >> shift) < bhi;
      const bool okv = ok && (v >> shift) >= blo && (v >> shift) < bhi;
      key[2 * i] = oku ? ((u << 32) | v) : ~0ull;
      key[2 * i + 1] = okv ? ((v << 32) | u) : ~0ull;
      if (oku) slot[2 * i] = atomicAdd(&lcnt[u >> shift], 1u);
      if (okv) slot[2 * i + 1] = atomicAdd(&lcnt[v >> shift], 1u);
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < nbk; b += kB)
      if (lcnt[b]) lbase[b] = atomicAdd(&cursor[b], (unsigned long long)lcnt[b]);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2 * kPer; ++i) {
      if (key[i] != ~0ull) {
        const uint32_t b = (uint32_t)((key[i] >> 32) >> shift);
        keys[lbase[b] + slot[i]] = key[i];
      }
    }
    __syncthreads();
  }
}

Src make_rmat(uint32_t scale, uint64_t seed, uint32_t ta, uint32_t tab,
              uint32_t tabc) {
  Src S{};
  S.kind = 0;
  S.scale = scale;
  S.ta = ta;
  S.tab = tab;
  S.tabc = tabc;
  S.state = gen_state(seed, GEN_TAG_RMAT);
  S.perm = gen_make_perm(seed, scale);
  return S;
}

Src make_chunglu(uint32_t n, uint64_t seed, const uint64_t* thr,
                 const uint32_t* alias) {
  Src S{};
  S.kind = 1;
  S.n = n;
  S.state = gen_state(seed, GEN_TAG_CHUNGLU);
  S.thr = thr;
  S.alias = alias;
  return S;
}

int launch(const Src& S, int phase, uint64_t s0, uint64_t cnt, uint32_t shift,
           uint32_t nbk, uint32_t blo, uint32_t bhi, unsigned long long* arr,
           uint64_t* keys, void* stream) {
  if (nbk == 0 || nbk > kMaxBuckets) return -1;
  uint64_t blocks = (cnt + kB - 1) / kB;
  if (blocks > 16384) blocks = 16384;
  if (blocks == 0) blocks = 1;
  hipStream_t st = (hipStream_t)stream;
  if (phase == 0)
    hipLaunchKernelGGL(k_count, dim3((uint32_t)blocks), dim3(kB), 0, st, S, s0, cnt,
                       shift, nbk, arr);
  else
    hipLaunchKernelGGL(k_scatter, dim3((uint32_t)blocks), dim3(kB), 0, st, S, s0,
                       cnt, shift, nbk, blo, bhi, arr, keys);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // namespace

extern "C" {

// phase 0: counts[b] += number of keys with source bucket b (u >> shift);
// phase 1: keys[cursor[b]++] = key for every key of a bucket b in
// [blo, bhi) (keys of other buckets are skipped).
int gen_rmat_gpu(int phase, uint32_t scale, uint64_t seed, uint32_t ta,
                 uint32_t tab, uint32_t tabc, uint64_t s0, uint64_t cnt,
                 uint32_t shift, uint32_t nbk, uint32_t blo, uint32_t bhi,
                 unsigned long long* arr, uint64_t* keys, void* stream) {
  return launch(make_rmat(scale, seed, ta, tab, tabc), phase, s0, cnt, shift, nbk,
                blo, bhi, arr, keys, stream);
}

int gen_chunglu_gpu(int phase, uint32_t n, uint64_t seed, const uint64_t* thr,
                    const uint32_t* alias, uint64_t s0, uint64_t cnt,
                    uint32_t shift, uint32_t nbk, uint32_t blo, uint32_t bhi,
                    unsigned long long* arr, uint64_t* keys, void* stream) {
  return launch(make_chunglu(n, seed, thr, alias), phase, s0, cnt, shift, nbk, blo,
                bhi, arr, keys, stream);
}

// Pinned host memory of exactly 'bytes' (the caller frees it).
void* gen_host_alloc(uint64_t bytes) {
  void* p = nullptr;
  if (hipHostMalloc(&p, bytes ? bytes : 8, hipHostMallocDefault) != hipSuccess) {
    (void)hipGetLastError();  // leave no error behind for the next HIP call
    return nullptr;
  }
  return p;
}

void gen_host_free(void* p) {
  if (p) (void)hipHostFree(p);
}

}  // extern "C"
