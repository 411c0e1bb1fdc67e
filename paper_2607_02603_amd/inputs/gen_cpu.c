/*
 * CPU build of the seeded graph samplers (see gen_common.h).  Samples are
 * written to fixed slots (2 keys per sample, UINT64_MAX for a dropped
 * self-loop) so the output does not depend on thread scheduling; the Python
 * side removes the sentinels, sorts, deduplicates and builds the CSR.
 * Key of a directed entry (u, v) = u << 32 | v.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "gen_common.h"

void gen_rmat_keys_cpu(uint32_t scale, uint64_t s_begin, uint64_t s_count,
                       uint64_t seed, uint32_t ta, uint32_t tab, uint32_t tabc,
                       uint64_t *keys)
{
    const uint64_t st = gen_state(seed, GEN_TAG_RMAT);
    const gen_perm pm = gen_make_perm(seed, scale);
#pragma omp parallel for schedule(static)
    for (int64_t q = 0; q < (int64_t)s_count; ++q) {
        uint64_t u, v;
        gen_rmat_raw(st, s_begin + (uint64_t)q, scale, ta, tab, tabc, &u, &v);
        u = gen_apply_perm(&pm, u);
        v = gen_apply_perm(&pm, v);
        if (u == v) {
            keys[2 * q] = UINT64_MAX;
            keys[2 * q + 1] = UINT64_MAX;
        } else {
            keys[2 * q] = (u << 32) | v;
            keys[2 * q + 1] = (v << 32) | u;
        }
    }
}

void gen_chunglu_keys_cpu(uint32_t n, uint64_t s_begin, uint64_t s_count,
                          uint64_t seed, const uint64_t *thr,
                          const uint32_t *alias, uint64_t *keys)
{
    const uint64_t st = gen_state(seed, GEN_TAG_CHUNGLU);
#pragma omp parallel for schedule(static)
    for (int64_t q = 0; q < (int64_t)s_count; ++q) {
        uint64_t s = s_begin + (uint64_t)q;
        uint64_t u = gen_alias_draw(gen_u64(st, 2 * s), n, thr, alias);
        uint64_t v = gen_alias_draw(gen_u64(st, 2 * s + 1), n, thr, alias);
        if (u == v) {
            keys[2 * q] = UINT64_MAX;
            keys[2 * q + 1] = UINT64_MAX;
        } else {
            keys[2 * q] = (u << 32) | v;
            keys[2 * q + 1] = (v << 32) | u;
        }
    }
}

/* Vose's alias method: thr[j] = round(prob_j * n * 2^32) in [0, 2^32]. */
int gen_alias_build(uint32_t n, const double *w, uint64_t *thr, uint32_t *alias)
{
    double sum = 0.0;
    for (uint32_t i = 0; i < n; ++i)
        sum += w[i];
    double *q = (double *)malloc((size_t)n * sizeof(double));
    uint32_t *small = (uint32_t *)malloc((size_t)n * sizeof(uint32_t));
    uint32_t *large = (uint32_t *)malloc((size_t)n * sizeof(uint32_t));
    if (!q || !small || !large)
        return -1;
    uint32_t ns = 0, nl = 0;
    for (uint32_t i = 0; i < n; ++i) {
        q[i] = w[i] * (double)n / sum;
        alias[i] = i;
        if (q[i] < 1.0)
            small[ns++] = i;
        else
            large[nl++] = i;
    }
    while (ns > 0 && nl > 0) {
        uint32_t s = small[--ns], l = large[--nl];
        thr[s] = (uint64_t)llround(q[s] * 4294967296.0);
        alias[s] = l;
        q[l] = (q[l] + q[s]) - 1.0;
        if (q[l] < 1.0)
            small[ns++] = l;
        else
            large[nl++] = l;
    }
    while (nl > 0) {
        uint32_t l = large[--nl];
        thr[l] = 4294967296ULL;
        alias[l] = l;
    }
    while (ns > 0) {
        uint32_t s = small[--ns];
        thr[s] = 4294967296ULL;
        alias[s] = s;
    }
    free(q);
    free(small);
    free(large);
    return 0;
}

/* G(n, m): the first m distinct unordered pairs {u, v}, u != v, of the
 * stream; u = hi32(U) * n >> 32, v = lo32(U) * n >> 32.  Returns the number
 * of stream values consumed.  out_u < out_v. */
uint64_t gen_er_edges(uint32_t n, uint64_t m, uint64_t seed, uint32_t *out_u,
                      uint32_t *out_v)
{
    const uint64_t st = gen_state(seed, GEN_TAG_ER);
    uint64_t cap = 16;
    while (cap < 4 * m)
        cap <<= 1;
    uint64_t *tab = (uint64_t *)malloc(cap * sizeof(uint64_t));
    for (uint64_t i = 0; i < cap; ++i)
        tab[i] = UINT64_MAX;
    uint64_t got = 0, i = 0;
    while (got < m) {
        uint64_t r = gen_u64(st, i++);
        uint32_t u = (uint32_t)(((r >> 32) * (uint64_t)n) >> 32);
        uint32_t v = (uint32_t)(((r & 0xFFFFFFFFULL) * (uint64_t)n) >> 32);
        if (u == v)
            continue;
        if (u > v) {
            uint32_t t = u;
            u = v;
            v = t;
        }
        uint64_t key = ((uint64_t)u << 32) | v;
        uint64_t h = gen_mix(key) & (cap - 1);
        int dup = 0;
        while (tab[h] != UINT64_MAX) {
            if (tab[h] == key) {
                dup = 1;
                break;
            }
            h = (h + 1) & (cap - 1);
        }
        if (dup)
            continue;
        tab[h] = key;
        out_u[got] = u;
        out_v[got] = v;
        ++got;
    }
    free(tab);
    return i;
}
