/*
 * CPU oracle for randomized 1-WL stable coloring — TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark may load this code.  The product path (the HIP library) never
 * calls, links or includes it, and this file shares no code with it.
 *
 * Everything here is written to be slow and obviously correct:
 *   - modular sums are accumulated exactly in 128-bit integers and reduced
 *     with the C '%' operator at the end;
 *   - the relabel is a plain qsort of (old color, image) pairs followed by a
 *     walk that hands out ranks;
 *   - classic refinement builds every node's full neighbour-colour multiset;
 *   - splitter refinement (oracle (b'), at the end of this file) reaches the
 *     coarsest stable colouring without rounds or random values, by a work
 *     list of splitter classes over the transpose.
 *
 * Paper: "Scaling Weisfeiler-Leman Expressiveness Analysis to Massive Graphs
 * with GPUs" (Biondi, Tribastone, Tschaikowski).  Section and equation names
 * below refer to it.
 *
 * Readings where the paper leaves a choice open (each is listed in the design
 * notes of the repository):
 *   - two arithmetics for the image z = A w, chosen by the argument q of the
 *     *_q functions:
 *       q = 0  (ORC_FP, the default): the prime field F_p, p = 2^61 - 1, in
 *              place of the ring of Section 4.1 (a nonzero linear form over a
 *              field vanishes on a uniform probe with probability exactly
 *              1/p, so the resampling step "until |H| distinct values" of
 *              Algorithm 1 is not needed and not done);
 *       q = 64 (ORC_RING64): the ring R = Z/2^64 of Section 4.1 and
 *              Algorithm 1 with precision q = 64: unsigned 64-bit values,
 *              sums and products taken modulo 2^64.  The resampling step is
 *              kept as a check: the k values of a round must be pairwise
 *              distinct.  They always are (the SplitMix64 output function is
 *              a bijection of 64-bit words and the k stream states are
 *              distinct), so one draw suffices.  Theorem 1's preconditions,
 *              n <= 2^32 and every row sum <= 2^32, are checked first;
 *   - the per-colour random value of colour b in round r is
 *     W(seed, r, b) = (b+1)-th output of a SplitMix64 stream whose state is
 *     K(seed, r) = mix(mix(seed + g) + (r+1) g), reduced mod p in F_p and
 *     taken as it is in Z/2^64
 *     (SplitMix64: Steele, Lea, Flood, OOPSLA 2014; the paper's appendix
 *     seeds its generator with SplitMix64 as well);
 *   - the new colour of node i is the rank of the pair (c_i, z_i) among the
 *     distinct pairs in lexicographic order (the "lexicographic sort" of
 *     Section 4.1 and of the proof of Theorem 1);
 *   - 'rounds' counts every SpMV + relabel round including the last one,
 *     which confirms that nothing split;
 *   - an empty row gives z_i = 0 (no A + I in the unbatched algorithm).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define ORC_P ((uint64_t)0x1FFFFFFFFFFFFFFFULL) /* 2^61 - 1 */
#define ORC_GAMMA ((uint64_t)0x9E3779B97F4A7C15ULL)

/* ------------------------------------------------------------------------- */
/* SplitMix64 (Steele, Lea, Flood 2014): output function and the weights.     */
/* ------------------------------------------------------------------------- */

uint64_t orc_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * (uint64_t)0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * (uint64_t)0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* i-th output (i = 1, 2, ...) of a SplitMix64 stream started from 'state'. */
uint64_t orc_splitmix_nth(uint64_t state, uint64_t i)
{
    return orc_mix64(state + i * ORC_GAMMA);
}

/* Per-round stream state K(seed, r): first output of a stream seeded with
 * 'seed' used as the state of a second stream, advanced r+1 steps. */
uint64_t orc_round_key(uint64_t seed, uint64_t round)
{
    uint64_t s1 = orc_splitmix_nth(seed, 1);
    return orc_splitmix_nth(s1, round + 1);
}

#define ORC_FP 0     /* arithmetic in F_p, p = 2^61 - 1 */
#define ORC_RING64 64 /* arithmetic in Z/2^64 (Algorithm 1, q = 64) */

/* Random value of colour b in round r (Algorithm 1: one value per block). */
uint64_t orc_weight_q(uint64_t seed, uint64_t round, uint64_t color, uint32_t q)
{
    uint64_t v = orc_splitmix_nth(orc_round_key(seed, round), color + 1);
    return q == ORC_RING64 ? v : v % ORC_P;
}

uint64_t orc_weight(uint64_t seed, uint64_t round, uint64_t color)
{
    return orc_weight_q(seed, round, color, ORC_FP);
}

static int cmp_u64(const void *a, const void *b)
{
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return (x > y) - (x < y);
}

/* Theorem 1's preconditions for Z/2^q: n <= 2^(q/2) and every row sum of A
 * at most 2^(q/2).  Returns 1 when they hold (q = 64). */
int orc_ring_preconditions(uint64_t n, const uint64_t *row_ptr,
                           const uint32_t *weight)
{
    const u128 lim = (u128)1 << 32;
    if (n > (uint64_t)lim)
        return 0;
    for (uint64_t i = 0; i < n; ++i) {
        u128 s = 0;
        for (uint64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
            s += weight ? weight[e] : 1;
        if (s > lim)
            return 0;
    }
    return 1;
}

/* ------------------------------------------------------------------------- */
/* Canonical initial colouring: dense rank of each label among the distinct   */
/* labels (order preserving).  NULL labels mean the trivial partition.        */
/* ------------------------------------------------------------------------- */

static int cmp_u32(const void *a, const void *b)
{
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return (x > y) - (x < y);
}

uint32_t orc_canonicalize(uint64_t n, const uint32_t *labels, uint32_t *out)
{
    if (n == 0)
        return 0;
    if (!labels) {
        for (uint64_t i = 0; i < n; ++i)
            out[i] = 0;
        return 1;
    }
    uint32_t *s = (uint32_t *)malloc(n * sizeof(uint32_t));
    memcpy(s, labels, n * sizeof(uint32_t));
    qsort(s, n, sizeof(uint32_t), cmp_u32);
    uint64_t k = 0;
    for (uint64_t i = 0; i < n; ++i)
        if (i == 0 || s[i] != s[i - 1])
            s[k++] = s[i];
    for (uint64_t i = 0; i < n; ++i) {
        uint64_t lo = 0, hi = k; /* first index with s[idx] >= labels[i] */
        while (lo < hi) {
            uint64_t mid = (lo + hi) / 2;
            if (s[mid] < labels[i])
                lo = mid + 1;
            else
                hi = mid;
        }
        out[i] = (uint32_t)lo;
    }
    free(s);
    return (uint32_t)k;
}

/* ------------------------------------------------------------------------- */
/* Oracle (a): one randomized round of Algorithm 1.                           */
/* ------------------------------------------------------------------------- */

typedef struct {
    uint32_t c;
    uint32_t node;
    uint64_t z;
} orc_pair;

static int cmp_pair(const void *a, const void *b)
{
    const orc_pair *x = (const orc_pair *)a, *y = (const orc_pair *)b;
    if (x->c != y->c)
        return (x->c > y->c) - (x->c < y->c);
    return (x->z > y->z) - (x->z < y->z);
}

/* z = A w where w_j = W(seed, round, c_j), in F_p (q = 0) or in Z/2^64
 * (q = 64).  A is CSR (row_ptr has n+1 entries; weight == NULL means every
 * stored entry has weight 1).  The sums are exact in 128 bits and reduced
 * once.  Returns 0, -1 if (q = 64) the k values are not pairwise distinct
 * (the repeat-until condition of Algorithm 1; it does not happen, see the
 * header), -2 for an unknown q. */
int orc_image_q(uint64_t n, const uint64_t *row_ptr, const uint32_t *col,
                const uint32_t *weight, const uint32_t *c, uint32_t k,
                uint64_t seed, uint64_t round, uint64_t *z, uint32_t q)
{
    if (q != ORC_FP && q != ORC_RING64)
        return -2;
    uint64_t *w = (uint64_t *)malloc((k ? k : 1) * sizeof(uint64_t));
    for (uint32_t b = 0; b < k; ++b)
        w[b] = orc_weight_q(seed, round, b, q);
    if (q == ORC_RING64 && k > 1) {
        uint64_t *s = (uint64_t *)malloc(k * sizeof(uint64_t));
        memcpy(s, w, k * sizeof(uint64_t));
        qsort(s, k, sizeof(uint64_t), cmp_u64);
        int dup = 0;
        for (uint32_t b = 1; b < k; ++b)
            dup |= s[b] == s[b - 1];
        free(s);
        if (dup) {
            free(w);
            return -1;
        }
    }
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        u128 acc = 0;
        for (uint64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            uint64_t a = weight ? weight[e] : 1;
            acc += (u128)a * w[c[col[e]]];
        }
        z[i] = q == ORC_RING64 ? (uint64_t)acc : (uint64_t)(acc % ORC_P);
    }
    free(w);
    return 0;
}

void orc_image(uint64_t n, const uint64_t *row_ptr, const uint32_t *col,
               const uint32_t *weight, const uint32_t *c, uint32_t k,
               uint64_t seed, uint64_t round, uint64_t *z)
{
    orc_image_q(n, row_ptr, col, weight, c, k, seed, round, z, ORC_FP);
}

/* New colour = rank of (c_i, z_i) among distinct pairs, lexicographic. */
uint32_t orc_relabel(uint64_t n, const uint32_t *c, const uint64_t *z,
                     uint32_t *c_out)
{
    if (n == 0)
        return 0;
    orc_pair *pr = (orc_pair *)malloc(n * sizeof(orc_pair));
    for (uint64_t i = 0; i < n; ++i) {
        pr[i].c = c[i];
        pr[i].z = z[i];
        pr[i].node = (uint32_t)i;
    }
    qsort(pr, n, sizeof(orc_pair), cmp_pair);
    uint64_t rank = 0;
    for (uint64_t t = 0; t < n; ++t) {
        if (t > 0 && cmp_pair(&pr[t - 1], &pr[t]) != 0)
            ++rank;
        c_out[pr[t].node] = (uint32_t)rank;
    }
    free(pr);
    return (uint32_t)(rank + 1);
}

/* One full round; returns k' (0 if the image step failed, see orc_image_q).
 * z may be NULL (scratch is allocated then). */
uint32_t orc_refine_round_q(uint64_t n, const uint64_t *row_ptr,
                            const uint32_t *col, const uint32_t *weight,
                            const uint32_t *c_in, uint32_t k_in, uint64_t seed,
                            uint64_t round, uint32_t *c_out, uint64_t *z_out,
                            uint32_t q)
{
    if (n == 0)
        return 0;
    uint64_t *z = z_out ? z_out : (uint64_t *)malloc(n * sizeof(uint64_t));
    uint32_t k = 0;
    if (orc_image_q(n, row_ptr, col, weight, c_in, k_in, seed, round, z, q) == 0)
        k = orc_relabel(n, c_in, z, c_out);
    if (!z_out)
        free(z);
    return k;
}

uint32_t orc_refine_round(uint64_t n, const uint64_t *row_ptr,
                          const uint32_t *col, const uint32_t *weight,
                          const uint32_t *c_in, uint32_t k_in, uint64_t seed,
                          uint64_t round, uint32_t *c_out, uint64_t *z_out)
{
    return orc_refine_round_q(n, row_ptr, col, weight, c_in, k_in, seed, round,
                              c_out, z_out, ORC_FP);
}

/* Algorithm 1 to completion.  Returns 0 on success, 1 if max_rounds was hit
 * (then c_out holds the last round's colours), 3 if q = 64 and Theorem 1's
 * preconditions fail (nothing is computed), 4 if an image step failed.
 * k_hist (may be NULL) receives the colour count after each round (capacity
 * max_rounds). */
int orc_stable_coloring_q(uint64_t n, const uint64_t *row_ptr,
                          const uint32_t *col, const uint32_t *weight,
                          const uint32_t *init, uint64_t seed,
                          uint32_t max_rounds, uint32_t *c_out, uint32_t *k_out,
                          uint32_t *rounds_out, uint32_t *k_hist, uint32_t q)
{
    *k_out = 0;
    *rounds_out = 0;
    if (q == ORC_RING64 && !orc_ring_preconditions(n, row_ptr, weight))
        return 3;
    if (n == 0)
        return 0;
    uint32_t *c = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t k = orc_canonicalize(n, init, c);
    int status = 1;
    uint32_t r = 0;
    while (r < max_rounds) {
        uint32_t k2 = orc_refine_round_q(n, row_ptr, col, weight, c, k, seed, r,
                                         c_out, NULL, q);
        if (k2 == 0) {
            status = 4;
            break;
        }
        if (k_hist)
            k_hist[r] = k2;
        ++r;
        memcpy(c, c_out, n * sizeof(uint32_t));
        if (k2 == k) {
            status = 0;
            break;
        }
        k = k2;
    }
    memcpy(c_out, c, n * sizeof(uint32_t));
    *k_out = k;
    *rounds_out = r;
    free(c);
    return status;
}

int orc_stable_coloring(uint64_t n, const uint64_t *row_ptr,
                        const uint32_t *col, const uint32_t *weight,
                        const uint32_t *init, uint64_t seed,
                        uint32_t max_rounds, uint32_t *c_out, uint32_t *k_out,
                        uint32_t *rounds_out, uint32_t *k_hist)
{
    return orc_stable_coloring_q(n, row_ptr, col, weight, init, seed, max_rounds,
                                 c_out, k_out, rounds_out, k_hist, ORC_FP);
}

/* ------------------------------------------------------------------------- */
/* Oracle (b): classic exact colour refinement.  Signature of node i is        */
/* (c_i, sorted list of (colour, total weight) over its out-neighbours); the   */
/* new colour is the dense rank of the signature (full-key comparison).        */
/* ------------------------------------------------------------------------- */

typedef struct {
    uint32_t color;
    uint32_t pad;
    uint64_t wsum;
} orc_term;

static const uint32_t *g_sig_c;
static const uint64_t *g_sig_ptr;
static const orc_term *g_sig;

static int cmp_term(const void *a, const void *b)
{
    const orc_term *x = (const orc_term *)a, *y = (const orc_term *)b;
    return (x->color > y->color) - (x->color < y->color);
}

static int cmp_sig(const void *a, const void *b)
{
    uint32_t i = *(const uint32_t *)a, j = *(const uint32_t *)b;
    if (g_sig_c[i] != g_sig_c[j])
        return (g_sig_c[i] > g_sig_c[j]) - (g_sig_c[i] < g_sig_c[j]);
    uint64_t li = g_sig_ptr[i + 1] - g_sig_ptr[i];
    uint64_t lj = g_sig_ptr[j + 1] - g_sig_ptr[j];
    const orc_term *si = g_sig + g_sig_ptr[i], *sj = g_sig + g_sig_ptr[j];
    uint64_t l = li < lj ? li : lj;
    for (uint64_t t = 0; t < l; ++t) {
        if (si[t].color != sj[t].color)
            return (si[t].color > sj[t].color) - (si[t].color < sj[t].color);
        if (si[t].wsum != sj[t].wsum)
            return (si[t].wsum > sj[t].wsum) - (si[t].wsum < sj[t].wsum);
    }
    return (li > lj) - (li < lj);
}

/* One classic round: c_out = dense rank of the signatures; returns k'.
 * Signature terms whose weight sum is 0 are dropped (Definition "Stable
 * Coloring" compares a_{i,B}, which is 0 for an unreached block too). */
uint32_t orc_classic_round(uint64_t n, const uint64_t *row_ptr,
                           const uint32_t *col, const uint32_t *weight,
                           const uint32_t *c, uint32_t *c_out)
{
    if (n == 0)
        return 0;
    uint64_t m = row_ptr[n];
    orc_term *sig = (orc_term *)malloc((m ? m : 1) * sizeof(orc_term));
    uint64_t *sig_ptr = (uint64_t *)malloc((n + 1) * sizeof(uint64_t));
    /* Per node: collect (colour, weight), sort by colour, merge equal colours.
     * The merged list of node i is written compacted at row_ptr[i]; its
     * length is recorded and the lists are packed afterwards. */
    uint64_t *len = (uint64_t *)malloc(n * sizeof(uint64_t));
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        orc_term *s = sig + row_ptr[i];
        uint64_t d = row_ptr[i + 1] - row_ptr[i];
        for (uint64_t t = 0; t < d; ++t) {
            uint64_t e = row_ptr[i] + t;
            s[t].color = c[col[e]];
            s[t].pad = 0;
            s[t].wsum = weight ? weight[e] : 1;
        }
        qsort(s, d, sizeof(orc_term), cmp_term);
        uint64_t u = 0;
        for (uint64_t t = 0; t < d; ++t) {
            if (u > 0 && s[u - 1].color == s[t].color)
                s[u - 1].wsum += s[t].wsum;
            else
                s[u++] = s[t];
        }
        /* a block reached with total weight 0 is the same as a block not
         * reached: the definition compares the sums a_{i,B} only */
        uint64_t kept = 0;
        for (uint64_t t = 0; t < u; ++t)
            if (s[t].wsum != 0)
                s[kept++] = s[t];
        len[i] = kept;
    }
    /* pack (in place, moving left only) */
    sig_ptr[0] = 0;
    for (uint64_t i = 0; i < n; ++i) {
        uint64_t src = row_ptr[i], dst = sig_ptr[i];
        if (src != dst)
            memmove(sig + dst, sig + src, len[i] * sizeof(orc_term));
        sig_ptr[i + 1] = dst + len[i];
    }
    uint32_t *order = (uint32_t *)malloc(n * sizeof(uint32_t));
    for (uint64_t i = 0; i < n; ++i)
        order[i] = (uint32_t)i;
    g_sig_c = c;
    g_sig_ptr = sig_ptr;
    g_sig = sig;
    qsort(order, n, sizeof(uint32_t), cmp_sig);
    uint64_t rank = 0;
    for (uint64_t t = 0; t < n; ++t) {
        if (t > 0 && cmp_sig(&order[t - 1], &order[t]) != 0)
            ++rank;
        c_out[order[t]] = (uint32_t)rank;
    }
    free(order);
    free(len);
    free(sig_ptr);
    free(sig);
    return (uint32_t)(rank + 1);
}

/* Classic refinement to the fixed point.  Same conventions as
 * orc_stable_coloring (rounds include the confirming round). */
int orc_classic_coloring(uint64_t n, const uint64_t *row_ptr,
                         const uint32_t *col, const uint32_t *weight,
                         const uint32_t *init, uint32_t max_rounds,
                         uint32_t *c_out, uint32_t *k_out,
                         uint32_t *rounds_out, uint32_t *k_hist)
{
    *k_out = 0;
    *rounds_out = 0;
    if (n == 0)
        return 0;
    uint32_t *c = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t k = orc_canonicalize(n, init, c);
    int status = 1;
    uint32_t r = 0;
    while (r < max_rounds) {
        uint32_t k2 = orc_classic_round(n, row_ptr, col, weight, c, c_out);
        if (k_hist)
            k_hist[r] = k2;
        ++r;
        memcpy(c, c_out, n * sizeof(uint32_t));
        if (k2 == k) {
            status = 0;
            break;
        }
        k = k2;
    }
    memcpy(c_out, c, n * sizeof(uint32_t));
    *k_out = k;
    *rounds_out = r;
    free(c);
    return status;
}

/* Exact stability certificate (Definition "Stable Coloring"): returns 0 when
 * every two nodes of a block have equal total out-weight into every block,
 * 1 otherwise.  'c' must be a dense colouring with k colours. */
int orc_is_stable(uint64_t n, const uint64_t *row_ptr, const uint32_t *col,
                  const uint32_t *weight, const uint32_t *c, uint32_t k)
{
    if (n == 0)
        return 0;
    uint32_t *tmp = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t k2 = orc_classic_round(n, row_ptr, col, weight, c, tmp);
    free(tmp);
    return k2 == k ? 0 : 1;
}

/* Relabel a colouring by first occurrence in node order (node 0 gets 0, each
 * new colour the next id).  Returns the number of colours. */
uint32_t orc_first_occurrence(uint64_t n, const uint32_t *c, uint32_t *out)
{
    if (n == 0)
        return 0;
    uint32_t mx = 0;
    for (uint64_t i = 0; i < n; ++i)
        if (c[i] > mx)
            mx = c[i];
    uint32_t *map = (uint32_t *)malloc(((uint64_t)mx + 1) * sizeof(uint32_t));
    for (uint64_t t = 0; t <= mx; ++t)
        map[t] = UINT32_MAX;
    uint32_t next = 0;
    for (uint64_t i = 0; i < n; ++i) {
        if (map[c[i]] == UINT32_MAX)
            map[c[i]] = next++;
        out[i] = map[c[i]];
    }
    free(map);
    return next;
}

/* ------------------------------------------------------------------------- */
/* Batched oracle: Algorithm 2 (Section 4.2) written out step by step.         */
/*                                                                             */
/* Readings: batches are greedy contiguous ranges of the CSR entry array that  */
/* end at a row boundary whenever the row fits, otherwise a row longer than    */
/* the cap is cut into pieces (its node is then a boundary node).  An empty    */
/* row belongs to the batch whose entry range contains its start offset (the   */
/* last batch when it sits at the very end), which avoids the footnote's A + I */
/* and the vacuous "inner to every batch".  Batch k of outer iteration t runs  */
/* Algorithm 1 with seed mix(seed + (2^32 t + k + 1) g).  The quotient uses the */
/* smallest node of each block as representative (Definition "Quotient        */
/* Graph" allows any); quotient nodes are numbered by first occurrence.        */
/* ------------------------------------------------------------------------- */

typedef struct {
    uint64_t tgt; /* target block */
    uint64_t w;
} orc_qent;

static int cmp_qent(const void *a, const void *b)
{
    const orc_qent *x = (const orc_qent *)a, *y = (const orc_qent *)b;
    return (x->tgt > y->tgt) - (x->tgt < y->tgt);
}

/* Batch boundaries in entry space: fills starts[] (capacity cap) and returns
 * the number of batches.  Batch b covers entries [starts[b], starts[b+1]) with
 * starts[nb] = m. */
uint64_t orc_batch_cut(uint64_t n, const uint64_t *row_ptr, uint64_t max_batch,
                       uint64_t *starts, uint64_t cap)
{
    uint64_t m = row_ptr[n];
    uint64_t nb = 0, s = 0, row = 0;
    if (max_batch == 0)
        return 0;
    do {
        if (nb < cap)
            starts[nb] = s;
        ++nb;
        if (m - s <= max_batch) {
            s = m;
            break;
        }
        /* advance 'row' to the last row boundary <= s + max_batch */
        uint64_t lim = s + max_batch;
        while (row < n && row_ptr[row + 1] <= lim)
            ++row;
        uint64_t e = row_ptr[row];
        if (e <= s)
            e = lim; /* the row at s does not fit: cut inside it */
        s = e;
    } while (s < m);
    if (nb < cap)
        starts[nb] = m;
    return nb;
}

/* Returns 0, 1 (a batch hit max_rounds), 2 (a quotient weight overflowed),
 * 3 (q = 64 and Theorem 1's preconditions fail; a quotient row sums the
 * same entries as its representative's row, so checking the input covers
 * every quotient) or 4 (an image step failed).
 *
 * early_stop != 0 adds the termination of Section 5.4 ("Feasibility"): once
 * the quotient of an outer iteration is built, the outer loop ends when that
 * quotient, cut with the same cap, would not give fewer batches than the
 * iteration just done (N_b counted as the ranges orc_batch_cut produces).
 * The colouring returned is then the merged partition of that iteration,
 * and the coarsest flag is 0 (several batches were used). */
int orc_batched_coloring_q(uint64_t n0, const uint64_t *row_ptr0,
                           const uint32_t *col0, const uint32_t *weight0,
                           const uint32_t *init, uint64_t seed,
                           uint64_t max_batch, uint32_t max_rounds,
                           uint32_t *c_out, uint32_t *k_out,
                           uint32_t *rounds_out, uint32_t *outer_out,
                           int *coarsest_out, uint32_t q, int early_stop)
{
    *k_out = 0;
    *rounds_out = 0;
    *outer_out = 0;
    *coarsest_out = 1;
    if (q == ORC_RING64 && !orc_ring_preconditions(n0, row_ptr0, weight0))
        return 3;
    if (n0 == 0)
        return 0;
    /* current graph (owned copies) */
    uint64_t n = n0;
    uint64_t *rp = (uint64_t *)malloc((n + 1) * sizeof(uint64_t));
    memcpy(rp, row_ptr0, (n + 1) * sizeof(uint64_t));
    uint64_t m = rp[n];
    uint32_t *col = (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t));
    memcpy(col, col0, m * sizeof(uint32_t));
    uint32_t *wt = (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t));
    for (uint64_t e = 0; e < m; ++e)
        wt[e] = weight0 ? weight0[e] : 1;
    uint32_t *label = (uint32_t *)malloc(n * sizeof(uint32_t));
    orc_canonicalize(n, init, label);
    uint32_t *map = (uint32_t *)malloc(n0 * sizeof(uint32_t));
    for (uint64_t i = 0; i < n0; ++i)
        map[i] = (uint32_t)i;
    uint32_t rounds_total = 0, outer = 0;
    int status = 0;

    for (uint64_t t = 0;; ++t) {
        m = rp[n];
        uint64_t nb = orc_batch_cut(n, rp, max_batch, NULL, 0);
        uint64_t *starts = (uint64_t *)malloc((nb + 1) * sizeof(uint64_t));
        orc_batch_cut(n, rp, max_batch, starts, nb + 1);
        /* batch label of each node: -1 = boundary */
        int64_t *owner = (int64_t *)malloc(n * sizeof(int64_t));
        for (uint64_t i = 0; i < n; ++i) {
            uint64_t a = rp[i], b = rp[i + 1];
            /* batch containing entry offset a (or the last batch if a == m) */
            uint64_t lo = 0, hi = nb - 1; /* last batch starting at or before a */
            while (lo < hi) {
                uint64_t mid = (lo + hi + 1) / 2;
                if (starts[mid] <= a)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            if (a == b)
                owner[i] = (int64_t)lo; /* empty row */
            else
                owner[i] = (b <= starts[lo + 1]) ? (int64_t)lo : -1;
        }
        /* merged partition: key per node, then first-occurrence ids */
        int64_t *key = (int64_t *)malloc(n * sizeof(int64_t));
        for (uint64_t i = 0; i < n; ++i)
            key[i] = -1;
        uint32_t *hc = (uint32_t *)malloc(n * sizeof(uint32_t));
        uint32_t *hout = (uint32_t *)malloc(n * sizeof(uint32_t));
        uint64_t *brp = (uint64_t *)malloc((n + 1) * sizeof(uint64_t));
        uint64_t block_base = 0;
        for (uint64_t b = 0; b < nb; ++b) {
            uint64_t s = starts[b], e = starts[b + 1];
            /* restricted graph A|E_b: all n rows, only entries in [s, e) */
            for (uint64_t i = 0; i <= n; ++i) {
                uint64_t v = rp[i];
                brp[i] = (v < s ? s : (v > e ? e : v)) - s;
            }
            /* H0_b: inner nodes keep their label class, others singletons */
            uint32_t *lab = hc;
            uint64_t nin = 0;
            uint32_t kin = 0;
            {
                /* dense ranks of the labels present among inner nodes */
                uint32_t *pres = (uint32_t *)calloc(n, sizeof(uint32_t));
                for (uint64_t i = 0; i < n; ++i)
                    if (owner[i] == (int64_t)b)
                        pres[label[i]] = 1;
                for (uint64_t v = 0; v < n; ++v) {
                    uint32_t f = pres[v];
                    pres[v] = kin;
                    kin += f;
                }
                uint32_t next = kin;
                for (uint64_t i = 0; i < n; ++i) {
                    if (owner[i] == (int64_t)b) {
                        lab[i] = pres[label[i]];
                        ++nin;
                    } else {
                        lab[i] = next++;
                    }
                }
                free(pres);
            }
            uint32_t kb = 0, rb = 0;
            uint64_t s_tb = orc_splitmix_nth(seed, (t << 32) + b + 1);
            int st = orc_stable_coloring_q(n, brp, col + s, wt + s, lab, s_tb,
                                           max_rounds, hout, &kb, &rb, NULL, q);
            rounds_total += rb;
            if (st == 4)
                status = 4;
            else if (st && status != 4)
                status = 1;
            for (uint64_t i = 0; i < n; ++i)
                if (owner[i] == (int64_t)b)
                    key[i] = (int64_t)(block_base + hout[i]);
            block_base += kb;
            (void)nin;
        }
        /* boundary nodes: singletons with fresh keys */
        for (uint64_t i = 0; i < n; ++i)
            if (key[i] < 0)
                key[i] = (int64_t)(block_base + i);
        /* first-occurrence block ids */
        uint64_t kmax = block_base + n;
        uint32_t *bid = (uint32_t *)malloc(kmax * sizeof(uint32_t));
        for (uint64_t v = 0; v < kmax; ++v)
            bid[v] = UINT32_MAX;
        uint32_t nq = 0;
        uint32_t *blk = hc; /* reuse */
        for (uint64_t i = 0; i < n; ++i) {
            if (bid[key[i]] == UINT32_MAX)
                bid[key[i]] = nq++;
            blk[i] = bid[key[i]];
        }
        free(bid);
        ++outer;
        /* compose the node -> block map */
        for (uint64_t i = 0; i < n0; ++i)
            map[i] = blk[map[i]];
        int last = (nb == 1) || (nq == n);
        if (last) {
            *coarsest_out = (nb == 1);
            free(starts);
            free(owner);
            free(key);
            free(hout);
            free(brp);
            free(hc);
            break;
        }
        /* quotient graph: row of block B = row of its smallest node, columns
         * mapped to blocks, weights summed per target block. */
        uint32_t *rep = (uint32_t *)malloc(nq * sizeof(uint32_t));
        for (uint64_t q = 0; q < nq; ++q)
            rep[q] = UINT32_MAX;
        for (uint64_t i = 0; i < n; ++i)
            if (rep[blk[i]] == UINT32_MAX)
                rep[blk[i]] = (uint32_t)i;
        uint64_t *qrp = (uint64_t *)malloc((nq + 1) * sizeof(uint64_t));
        uint64_t qm = 0;
        orc_qent *tmp = (orc_qent *)malloc((m ? m : 1) * sizeof(orc_qent));
        uint32_t *qcol = (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t));
        uint32_t *qwt = (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t));
        uint32_t *qlabel = (uint32_t *)malloc(nq * sizeof(uint32_t));
        qrp[0] = 0;
        for (uint64_t q = 0; q < nq; ++q) {
            uint32_t r = rep[q];
            uint64_t d = 0;
            for (uint64_t e = rp[r]; e < rp[r + 1]; ++e) {
                tmp[d].tgt = blk[col[e]];
                tmp[d].w = wt[e];
                ++d;
            }
            qsort(tmp, d, sizeof(orc_qent), cmp_qent);
            for (uint64_t t2 = 0; t2 < d; ++t2) {
                if (t2 > 0 && tmp[t2].tgt == tmp[t2 - 1].tgt) {
                    if ((uint64_t)qwt[qm - 1] + tmp[t2].w > UINT32_MAX)
                        status = 2; /* aggregated weight does not fit */
                    qwt[qm - 1] += (uint32_t)tmp[t2].w;
                } else {
                    qcol[qm] = (uint32_t)tmp[t2].tgt;
                    qwt[qm] = (uint32_t)tmp[t2].w;
                    ++qm;
                }
            }
            qrp[q + 1] = qm;
            qlabel[q] = label[r];
        }
        free(tmp);
        free(rep);
        free(rp);
        free(col);
        free(wt);
        free(label);
        rp = qrp;
        col = qcol;
        wt = qwt;
        label = qlabel;
        n = nq;
        free(starts);
        free(owner);
        free(key);
        free(hout);
        free(brp);
        free(hc);
        /* Section 5.4: stop when the next iteration would not have fewer
         * batches (nb > 1 here, else the loop ended above) */
        if (early_stop && orc_batch_cut(n, rp, max_batch, NULL, 0) >= nb) {
            *coarsest_out = 0;
            break;
        }
    }
    /* final colours: first occurrence over the original nodes */
    uint32_t k = orc_first_occurrence(n0, map, c_out);
    *k_out = k;
    *rounds_out = rounds_total;
    *outer_out = outer;
    free(map);
    free(rp);
    free(col);
    free(wt);
    free(label);
    return status;
}

int orc_batched_coloring(uint64_t n0, const uint64_t *row_ptr0,
                         const uint32_t *col0, const uint32_t *weight0,
                         const uint32_t *init, uint64_t seed,
                         uint64_t max_batch, uint32_t max_rounds,
                         uint32_t *c_out, uint32_t *k_out,
                         uint32_t *rounds_out, uint32_t *outer_out,
                         int *coarsest_out)
{
    return orc_batched_coloring_q(n0, row_ptr0, col0, weight0, init, seed,
                                  max_batch, max_rounds, c_out, k_out,
                                  rounds_out, outer_out, coarsest_out, ORC_FP, 0);
}

/* ------------------------------------------------------------------------- */
/* Oracle (b'): exact colour refinement by splitters.                          */
/*                                                                            */
/* The coarsest stable colouring refining the initial one (Definitions        */
/* "Stable Coloring" and "Coarsest Stable Coloring", Section 3), computed     */
/* the way the partition-refinement baselines the paper compares against     */
/* work (Section 2): a partition is stable exactly when, for every class S    */
/* (a splitter), all members i of a class C have the same weighted count      */
/* w(i, S) = sum of A[i][l] over l in S.  A work list holds the classes the   */
/* partition may not yet be stable against.  Taking S off the list, the       */
/* counts w(i, S) of every node with an entry into S are summed over the     */
/* transpose, and every class is split by them (members without such an      */
/* entry count 0).  When C splits into parts:                                 */
/*   - if C is on the list, every part is (C keeps its id on its first part); */
/*   - otherwise every part but one largest is listed: the partition was      */
/*     stable against C, and w(i, largest) = w(i, C) - sum of the others.     */
/* This is Hopcroft's "process the smaller half" (Hopcroft 1971), extended    */
/* to k-way splits of weighted counts by Cardon and Crochemore (1982) and     */
/* analysed for colour refinement by Berkholz, Bonsma and Grohe (2017): a     */
/* node lies in a processed splitter O(log n) times, so the entries are      */
/* visited O(m log n) times.  The touched members of a class are ordered by  */
/* a comparison sort here, which adds a logarithmic factor to that part.      */
/* Precondition: every weighted row sum fits in 64 bits (always true for     */
/* rows of fewer than 2^32 entries of 32-bit weights).                        */
/* ------------------------------------------------------------------------- */

typedef struct {
    uint64_t w;
    uint32_t node;
} orc_wnode;

/* ORC_PROGRESS=1 in the environment: progress lines on stderr (long runs). */
static int orc_progress_on(void)
{
    const char *s = getenv("ORC_PROGRESS");
    return s && s[0] == '1';
}

static int cmp_wnode(const void *a, const void *b)
{
    const orc_wnode *x = (const orc_wnode *)a, *y = (const orc_wnode *)b;
    if (x->w != y->w)
        return x->w < y->w ? -1 : 1;
    return (x->node > y->node) - (x->node < y->node);
}

/* Returns 0; c_out gets first-occurrence ids (node 0 has colour 0), k_out
 * the number of classes, visits_out (may be NULL) the number of transpose
 * entries read over all splitters. */
int orc_splitter_coloring(uint64_t n, const uint64_t *row_ptr,
                          const uint32_t *col, const uint32_t *weight,
                          const uint32_t *init, uint32_t *c_out,
                          uint32_t *k_out, uint64_t *visits_out)
{
    *k_out = 0;
    if (visits_out)
        *visits_out = 0;
    if (n == 0)
        return 0;
    const uint64_t m = row_ptr[n];
    /* transpose: for column l, the rows i with an entry A[i][l] */
    uint64_t *tptr = (uint64_t *)calloc(n + 1, sizeof(uint64_t));
    uint32_t *tsrc = (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t));
    uint32_t *twt = weight ? (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t)) : NULL;
    for (uint64_t e = 0; e < m; ++e)
        ++tptr[col[e] + 1];
    for (uint64_t l = 0; l < n; ++l)
        tptr[l + 1] += tptr[l];
    uint64_t *tfill = (uint64_t *)malloc(n * sizeof(uint64_t));
    memcpy(tfill, tptr, n * sizeof(uint64_t));
    for (uint64_t i = 0; i < n; ++i)
        for (uint64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            const uint64_t t = tfill[col[e]]++;
            tsrc[t] = (uint32_t)i;
            if (twt)
                twt[t] = weight[e];
        }
    free(tfill);
    const int prog = orc_progress_on();
    if (prog)
        fprintf(stderr, "[splitters] transpose built: n=%llu m=%llu\n",
                (unsigned long long)n, (unsigned long long)m);

    /* the partition: members of class c are elem[cbeg[c] .. cend[c]) */
    uint32_t *cls = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *elem = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *loc = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *cbeg = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *cend = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *cmark = (uint32_t *)calloc(n, sizeof(uint32_t)); /* touched members */
    uint8_t *listed = (uint8_t *)calloc(n, 1);
    uint32_t *work = (uint32_t *)malloc(n * sizeof(uint32_t)); /* the work list */
    uint32_t *touched = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *tclass = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint32_t *members = (uint32_t *)malloc(n * sizeof(uint32_t));
    uint64_t *cnt = (uint64_t *)calloc(n, sizeof(uint64_t));
    uint8_t *hit = (uint8_t *)calloc(n, 1);
    orc_wnode *tail = (orc_wnode *)malloc(n * sizeof(orc_wnode));

    uint32_t k = orc_canonicalize(n, init, cls);
    for (uint32_t c = 0; c < k; ++c)
        cbeg[c] = 0;
    {
        uint32_t *size = (uint32_t *)calloc(k, sizeof(uint32_t));
        for (uint64_t i = 0; i < n; ++i)
            ++size[cls[i]];
        uint32_t s = 0;
        for (uint32_t c = 0; c < k; ++c) {
            cbeg[c] = s;
            cend[c] = s;
            s += size[c];
        }
        free(size);
        for (uint64_t i = 0; i < n; ++i) {
            const uint32_t p = cend[cls[i]]++;
            elem[p] = (uint32_t)i;
            loc[i] = p;
        }
    }
    uint32_t nwork = 0;
    for (uint32_t c = 0; c < k; ++c) {
        work[nwork++] = c;
        listed[c] = 1;
    }
    uint64_t visits = 0, pmark = 0, npop = 0;
    while (nwork) {
        ++npop;
        const uint32_t s = work[--nwork];
        listed[s] = 0;
        /* the splitter's members as they are now */
        const uint32_t ns = cend[s] - cbeg[s];
        memcpy(members, elem + cbeg[s], ns * sizeof(uint32_t));
        uint32_t nt = 0, ntc = 0;
        for (uint32_t x = 0; x < ns; ++x) {
            const uint32_t l = members[x];
            for (uint64_t t = tptr[l]; t < tptr[l + 1]; ++t) {
                const uint32_t i = tsrc[t];
                ++visits;
                if (!hit[i]) {
                    /* move i to the touched tail of its class */
                    hit[i] = 1;
                    touched[nt++] = i;
                    const uint32_t c = cls[i];
                    if (cmark[c] == 0)
                        tclass[ntc++] = c;
                    const uint32_t dst = cend[c] - 1 - cmark[c]++;
                    const uint32_t other = elem[dst], src = loc[i];
                    elem[dst] = i;
                    loc[i] = dst;
                    elem[src] = other;
                    loc[other] = src;
                }
                cnt[i] += twt ? twt[t] : 1u;
            }
            if (prog && (visits >> 30) != pmark) {
                pmark = visits >> 30;
                fprintf(stderr, "[splitters] visits %llu, splitters %llu, classes %u, listed %u\n",
                        (unsigned long long)visits, (unsigned long long)npop, k, nwork);
            }
        }
        for (uint32_t y = 0; y < ntc; ++y) {
            const uint32_t c = tclass[y];
            const uint32_t b = cbeg[c], e = cend[c], nm = cmark[c];
            const uint32_t t0 = e - nm;
            cmark[c] = 0;
            for (uint32_t p = t0; p < e; ++p) {
                tail[p - t0].w = cnt[elem[p]];
                tail[p - t0].node = elem[p];
            }
            qsort(tail, nm, sizeof(orc_wnode), cmp_wnode);
            for (uint32_t p = t0; p < e; ++p) {
                elem[p] = tail[p - t0].node;
                loc[elem[p]] = p;
            }
            /* runs of equal counts in position order; the untouched
             * prefix [b, t0) counts 0, sorts first and is taken as one
             * run, so the walk costs only the touched members */
            uint32_t nruns = 0, big = 0, bigsize = 0;
            uint32_t p = b;
            while (p < e) {
                const uint64_t v = p < t0 ? 0 : tail[p - t0].w;
                uint32_t q = p < t0 ? t0 : p + 1;
                while (q < e && tail[q - t0].w == v)
                    ++q;
                if (q - p > bigsize) {
                    bigsize = q - p;
                    big = nruns;
                }
                ++nruns;
                p = q;
            }
            if (nruns == 1)
                continue;
            const int was_listed = listed[c];
            uint32_t r = 0;
            p = b;
            while (p < e) {
                const uint64_t v = p < t0 ? 0 : tail[p - t0].w;
                uint32_t q = p < t0 ? t0 : p + 1;
                while (q < e && tail[q - t0].w == v)
                    ++q;
                uint32_t id = c;
                if (r == 0) {
                    cend[c] = q;
                } else {
                    id = k++;
                    cbeg[id] = p;
                    cend[id] = q;
                    for (uint32_t z = p; z < q; ++z)
                        cls[elem[z]] = id;
                }
                if ((was_listed || r != big) && !listed[id]) {
                    work[nwork++] = id;
                    listed[id] = 1;
                }
                ++r;
                p = q;
            }
        }
        for (uint32_t x = 0; x < nt; ++x) {
            cnt[touched[x]] = 0;
            hit[touched[x]] = 0;
        }
    }
    *k_out = orc_first_occurrence(n, cls, c_out);
    if (visits_out)
        *visits_out = visits;
    free(tptr);
    free(tsrc);
    free(twt);
    free(cls);
    free(elem);
    free(loc);
    free(cbeg);
    free(cend);
    free(cmark);
    free(listed);
    free(work);
    free(touched);
    free(tclass);
    free(members);
    free(cnt);
    free(hit);
    free(tail);
    return 0;
}
