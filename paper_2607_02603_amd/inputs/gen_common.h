/*
 * Seeded synthetic graph samplers shared by the CPU (gcc) and GPU (hipcc)
 * builds of the input generators.  Only input generation lives here: nothing
 * of the colour-refinement method.  Every random number is a counter-based
 * SplitMix64 output, so sample s of a stream is the same on every device.
 *
 *   stream state   S(seed, tag) = mix(seed + tag * g)
 *   value i        U(S, i)      = mix(S + (i + 1) * g)
 *
 * R-MAT (Chakrabarti, Zhan, Faloutsos 2004; Graph500 convention): sample s
 * draws 'scale' quadrant choices, one per level from the most significant
 * bit down, each from a 32-bit uniform compared with the fixed-point
 * cumulative probabilities (a, a+b, a+b+c); two 32-bit uniforms per 64-bit
 * value, (scale+1)/2 values per sample.  Quadrant b sets the target bit,
 * c the source bit, d both.  Both endpoints then go through a seeded
 * bijection of [0, 2^scale) that scatters the hubs.
 *
 * Chung-Lu by edge sampling: both endpoints of sample s are drawn from an
 * alias table (Vose) of the weights w_i = (i + 1)^(-1/(gamma-1)) built on
 * the host; column j = hi32(U) * n >> 32, accepted if lo32(U) < thr[j],
 * else alias[j].
 */
#ifndef WL_GEN_COMMON_H
#define WL_GEN_COMMON_H
#include <stdint.h>

#ifdef __HIPCC__
#define GEN_FN __host__ __device__ __forceinline__
#else
#define GEN_FN static inline
#endif

#define GEN_GAMMA 0x9E3779B97F4A7C15ULL
#define GEN_TAG_ER 1ULL
#define GEN_TAG_CHUNGLU 2ULL
#define GEN_TAG_RMAT 3ULL
#define GEN_TAG_RMAT_PERM 4ULL

GEN_FN uint64_t gen_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

GEN_FN uint64_t gen_state(uint64_t seed, uint64_t tag)
{
    return gen_mix(seed + tag * GEN_GAMMA);
}

GEN_FN uint64_t gen_u64(uint64_t state, uint64_t i)
{
    return gen_mix(state + (i + 1) * GEN_GAMMA);
}

/* Parameters of the R-MAT vertex bijection. */
typedef struct {
    uint64_t m1, c1, m2, c2;
    uint32_t scale, sh1, sh2, pad;
} gen_perm;

GEN_FN gen_perm gen_make_perm(uint64_t seed, uint32_t scale)
{
    gen_perm p;
    uint64_t s = gen_state(seed, GEN_TAG_RMAT_PERM);
    p.m1 = gen_u64(s, 0) | 1ULL;
    p.c1 = gen_u64(s, 1);
    p.m2 = gen_u64(s, 2) | 1ULL;
    p.c2 = gen_u64(s, 3);
    p.scale = scale;
    p.sh1 = scale / 2 + 1;
    p.sh2 = (scale + 2) / 3 + 1;
    p.pad = 0;
    return p;
}

GEN_FN uint64_t gen_apply_perm(const gen_perm *p, uint64_t x)
{
    const uint64_t mask = (p->scale >= 64) ? ~0ULL : ((1ULL << p->scale) - 1);
    x = (x * p->m1 + p->c1) & mask;
    x ^= x >> p->sh1;
    x = (x * p->m2 + p->c2) & mask;
    x ^= x >> p->sh2;
    return x;
}

/* One R-MAT sample (before the bijection). */
GEN_FN void gen_rmat_raw(uint64_t state, uint64_t s, uint32_t scale,
                         uint32_t ta, uint32_t tab, uint32_t tabc,
                         uint64_t *u, uint64_t *v)
{
    const uint32_t words = (scale + 1) / 2;
    uint64_t uu = 0, vv = 0;
    for (uint32_t w = 0; w < words; ++w) {
        uint64_t r = gen_u64(state, s * words + w);
        for (uint32_t h = 0; h < 2; ++h) {
            uint32_t lvl = 2 * w + h;
            if (lvl >= scale)
                break;
            uint32_t x = (uint32_t)(h ? (r >> 32) : (r & 0xFFFFFFFFULL));
            uint64_t bu = (x >= tab) ? 1ULL : 0ULL;       /* c or d */
            uint64_t bv = (x >= ta && x < tab) || (x >= tabc) ? 1ULL : 0ULL;
            uu = (uu << 1) | bu;
            vv = (vv << 1) | bv;
        }
    }
    *u = uu;
    *v = vv;
}

/* Alias-table draw of one endpoint. */
GEN_FN uint32_t gen_alias_draw(uint64_t r, uint32_t n, const uint64_t *thr,
                               const uint32_t *alias)
{
    uint32_t j = (uint32_t)(((r >> 32) * (uint64_t)n) >> 32);
    return ((r & 0xFFFFFFFFULL) < thr[j]) ? j : alias[j];
}

#endif
