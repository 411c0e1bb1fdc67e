// Device-side helpers for the gfx950 kernels: arithmetic in F_p with
// p = 2^61 - 1 or in the ring Z/2^64, the SplitMix64 weight generator, and
// wave64 primitives.
//
// Method: randomized stable colouring (Algorithm 1, Section 4.1 of "Scaling
// Weisfeiler-Leman Expressiveness Analysis to Massive Graphs with GPUs").
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wl {

constexpr uint64_t kP = 0x1FFFFFFFFFFFFFFFull;      // 2^61 - 1
constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;  // SplitMix64 increment
constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// F_p arithmetic.  Residues are kept canonical in [0, p) wherever they are
// compared or stored.  Sums of many residues are accumulated in a 96-bit
// (lo:64, hi:32) register pair and folded once: 2^64 = 8 (mod p).
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint64_t fold61(uint64_t v) {
  // v < 2^64  ->  canonical residue of v mod p.
  uint64_t t = (v & kP) + (v >> 61);
  return t >= kP ? t - kP : t;
}

__device__ __forceinline__ uint64_t addp(uint64_t a, uint64_t b) {
  // a, b canonical.
  uint64_t s = a + b;
  return s >= kP ? s - kP : s;
}

struct Acc96 {
  uint64_t lo;
  uint32_t hi;
};

__device__ __forceinline__ void acc_add(Acc96& a, uint64_t v) {
  uint64_t s = a.lo + v;
  a.hi += (s < v) ? 1u : 0u;
  a.lo = s;
}

__device__ __forceinline__ uint64_t acc_reduce(const Acc96& a) {
  // value = hi * 2^64 + lo  ==  8 hi + (lo & p) + (lo >> 61)   (mod p)
  uint64_t t = (a.lo & kP) + (a.lo >> 61) + ((uint64_t)a.hi << 3);
  return fold61(t);
}

// a * x mod p folded to < 2^62 (not canonical) for a < 2^32, x < 2^61.
__device__ __forceinline__ uint64_t mul_small_fold(uint32_t a, uint64_t x) {
  uint64_t lo = (uint64_t)a * x;
  uint64_t hi = __umul64hi((uint64_t)a, x);
  return (lo & kP) + ((hi << 3) | (lo >> 61));
}

// a * b mod p for canonical a, b.
__device__ __forceinline__ uint64_t mulp(uint64_t a, uint64_t b) {
  const uint64_t lo = a * b;
  const uint64_t hi = __umul64hi(a, b);
  return fold61((lo & kP) + ((hi << 3) | (lo >> 61)));
}

// ---------------------------------------------------------------------------
// SplitMix64 (Steele, Lea, Flood 2014) and the per-colour random values.
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// State of the stream that serves round r.
__device__ __forceinline__ uint64_t round_key(uint64_t seed, uint32_t r) {
  uint64_t s1 = mix64(seed + kGamma);
  return mix64(s1 + ((uint64_t)r + 1) * kGamma);
}

// Random value of colour c: (c+1)-th output of the round's stream, reduced
// mod p, or taken as it is in Z/2^64 (ring != 0).  The outputs for distinct
// c are distinct: the states key + (c+1) g differ (g is odd) and the output
// function is a bijection of 64-bit words.
__device__ __forceinline__ uint64_t color_weight(uint64_t key, uint32_t c, uint32_t ring) {
  const uint64_t m = mix64(key + ((uint64_t)c + 1) * kGamma);
  return ring ? m : fold61(m);
}

// Same stream, 64-bit colour id (ids >= 2^32 name the frozen singleton
// classes of nodes outside a batch).
__device__ __forceinline__ uint64_t color_weight64(uint64_t key, uint64_t c, uint32_t ring) {
  const uint64_t m = mix64(key + (c + 1) * kGamma);
  return ring ? m : fold61(m);
}

// ---------------------------------------------------------------------------
// The two arithmetics of the image z = A w.  ring == 0: F_p as above; the
// values are canonical residues.  ring != 0: Z/2^64 (Algorithm 1 with
// precision q = 64): values, sums and products wrap at 2^64.  An Acc96 sum
// holds the exact sum's low 64 bits in 'lo', which is its value in Z/2^64.
// 'ring' is the same for every thread of a launch.
// ---------------------------------------------------------------------------

// a * x for a weight a < 2^32: mod p folded to < 2^62 for x < 2^61, or mod 2^64.
__device__ __forceinline__ uint64_t mul_small_q(uint32_t a, uint64_t x, uint32_t ring) {
  return ring ? (uint64_t)a * x : mul_small_fold(a, x);
}

// Value of an accumulated sum: canonical residue, or the sum mod 2^64.
__device__ __forceinline__ uint64_t acc_value(const Acc96& a, uint32_t ring) {
  return ring ? a.lo : acc_reduce(a);
}

__device__ __forceinline__ uint64_t add_q(uint64_t a, uint64_t b, uint32_t ring) {
  return ring ? a + b : addp(a, b);
}

// d * w for an integer d < 2^61 (a degree) and a value w.
__device__ __forceinline__ uint64_t mul_int_q(uint64_t d, uint64_t w, uint32_t ring) {
  return ring ? d * w : mulp(fold61(d), w);
}

// ---------------------------------------------------------------------------
// wave64 helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ int lane_id() { return __lane_id(); }

template <int G>
__device__ __forceinline__ uint64_t group_sum_q(uint64_t v, uint32_t ring) {
  // Sum over aligned groups of G lanes (G | 64) of canonical residues, or
  // of values mod 2^64.
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) {
    uint64_t o = __shfl_xor(v, off, kWave);
    v = add_q(v, o, ring);
  }
  return v;
}

}  // namespace wl
