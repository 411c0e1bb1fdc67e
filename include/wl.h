/*
 * wl.h — C ABI of the MI355X (gfx950) library for randomized 1-WL stable
 * colouring (randomized linear-algebraic colour refinement).
 *
 * Method: "Scaling Weisfeiler-Leman Expressiveness Analysis to Massive Graphs
 * with GPUs" (Biondi, Tribastone, Tschaikowski).
 *   - Algorithm 1 (Randomized Stable Coloring, Section 4.1): per round, draw
 *     one random value per colour, take the image z = A w, and split every
 *     colour class by z.
 *   - Algorithm 2 (Randomized Batched Stable Coloring, Section 4.2): cut the
 *     edge set into batches, refine each batch with its boundary nodes frozen
 *     as singletons (Eq. batch-init), merge (Eq. merge), contract to the
 *     quotient graph (Definition "Quotient Graph", Eq. sc) and repeat.
 *
 * Arithmetic: exact modular arithmetic in F_p, p = 2^61 - 1 (the default),
 * or in the ring Z/2^64 of Section 4.1 (wl_set_precision).  The random
 * value of colour b in round r is W(seed, r, b): the (b+1)-th output of a
 * SplitMix64 stream whose state is mix(mix(seed + g) + (r+1) g), reduced
 * mod p in F_p and taken as it is in Z/2^64 (g = 0x9E3779B97F4A7C15, mix =
 * the SplitMix64 output function).
 * New colour of node i = rank of the pair (c_i, z_i) among all distinct pairs
 * in lexicographic order.  Rounds repeat until the colour count does not
 * change; the round that confirms this is counted.
 *
 * Conventions shared by every entry point
 *   - Graphs are CSR.  Row i lists the out-neighbours of node i (the
 *     stability condition of the paper is on out-weights).  Column order
 *     inside a row does not matter; repeated columns count with
 *     multiplicity.  Self-loops are allowed.
 *   - The caller owns every buffer it passes.  Device memory: no entry point
 *     allocates any; all device scratch space is the caller's 'workspace'
 *     (256-byte aligned), sized by the *_workspace_size() call of each entry
 *     point.  Host memory: the in-core entry points (wl_refine_round,
 *     wl_stable_coloring, wl_verify_stable) allocate none beyond a few
 *     bytes of bookkeeping; the out-of-core ones (wl_stable_coloring_streamed,
 *     wl_stable_coloring_batched) allocate page-locked staging buffers and
 *     pageable arrays, stated at each, and free them before returning.
 *     Streams and events: the in-core entry points create none, except with
 *     WL_GRAPH=1 in the environment, where a call creates a capture stream
 *     and HIP graph objects and destroys them before it returns; the
 *     out-of-core ones create copy streams and events for the call's
 *     duration.
 *   - All device work is enqueued on 'stream' (a hipStream_t; NULL = the
 *     null stream).  Entry points that return host scalars synchronise that
 *     stream before returning.
 *   - Return value: WL_OK (0) or a negative WL_E* code; wl_last_error() then
 *     gives a message (thread-local).  Outputs are defined only on WL_OK,
 *     except WL_EMAXROUNDS (see wl_stable_coloring).  No C++ exception ever
 *     crosses this interface.
 *   - Preconditions checked on the host: n < 2^32, nnz consistent with the
 *     row pointer, non-NULL pointers where required.  Set the environment
 *     variable WL_VALIDATE=1 to also check, on the device, that row pointers
 *     are non-decreasing and every column index is < n (costs one pass), and
 *     for a graph flagged WL_CSR_SYMMETRIC that the multisets of entries
 *     (i, j) and (j, i) agree (compared through sums of 64-bit hashes).
 *   - Row sums of the weights must stay below p (true for every graph with
 *     uint32 weights and fewer than 2^29 entries per row, and preserved by
 *     quotients); in Z/2^64 they must be at most 2^32 (checked).
 */
#ifndef WL_H
#define WL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WL_OK 0
#define WL_EINVAL (-1)      /* malformed arguments or graph                */
#define WL_EBUDGET (-2)     /* workspace smaller than required             */
#define WL_EOVERFLOW (-3)   /* n >= 2^32, a quotient weight overflowed, or
                               a row sum above 2^32 in Z/2^64             */
#define WL_EMAXROUNDS (-4)  /* round cap reached before stability          */
#define WL_ENOTSTABLE (-5)  /* wl_verify_stable: colouring is not stable   */
#define WL_EHIP (-6)        /* a HIP runtime call failed                   */
#define WL_ENOMEM (-7)      /* a host allocation of the library failed     */

/* CSR adjacency.  Exactly one of row_ptr32 / row_ptr64 is non-NULL; it has
 * n+1 entries, row_ptr[0] == 0 and row_ptr[n] == nnz.  col_idx has nnz
 * entries, each < n.  weight is NULL (every entry weighs 1) or has nnz
 * entries (a_ij in N_0; weighted graphs arise as quotients).  Whether the
 * pointers are device or host memory is stated per entry point.
 * flags: WL_CSR_SYMMETRIC states that A equals its transpose (every entry
 * (i, j) has a matching entry (j, i), multiplicities included), as for the
 * CSR of an undirected graph stored in both directions.  For an unweighted
 * symmetric graph with fewer than 2^32 entries the in-core entry points may
 * then compute A w by routing each row's value to its neighbours through
 * LDS-sized bins (streaming passes) instead of one random read per entry;
 * this needs the larger workspace wl_workspace_size() reports for such a
 * graph (about 8 bytes more per entry) and is skipped when the workspace is
 * smaller.  A graph flagged symmetric that is not is reported as WL_EINVAL
 * when the library notices (it checks the entry counts per bin of rows;
 * results are defined only for correctly flagged graphs). */
#define WL_CSR_SYMMETRIC 1ull
typedef struct wl_csr {
    uint64_t n;
    uint64_t nnz;
    const uint32_t *row_ptr32;
    const uint64_t *row_ptr64;
    const uint32_t *col_idx;
    const uint32_t *weight;
    uint64_t flags;
} wl_csr;

/* Workspace (device bytes) needed by the in-core entry points
 * (wl_refine_round, wl_stable_coloring) for graph g.
 * Only g->n, g->nnz, g->flags and whether g->weight is NULL are read; the
 * pointers may be NULL otherwise.
 * Returns WL_EINVAL for a NULL argument, WL_EOVERFLOW for n >= 2^32. */
int wl_workspace_size(const wl_csr *g, uint64_t *bytes_out);

/* Smallest workspace accepted by wl_stable_coloring_batched for a graph
 * with g->n nodes: the node-sized state plus room for a batch of
 * 'max_batch_entries' CSR entries (pass 0 to ask for the size that holds the
 * whole graph in one batch). */
int wl_batched_workspace_size(const wl_csr *g, uint64_t max_batch_entries,
                              uint64_t *bytes_out);

/* One round of Algorithm 1 (Section 4.1).
 *   g          device CSR.
 *   color_in   device, n entries, each < k_in (a colouring; ids need not all
 *              be used).  k_in <= max(n, 1).
 *   seed,round select the random values W(seed, round, .).
 *   color_out  device, n entries; receives the rank of (color_in[i], z_i)
 *              among the distinct pairs.  May alias color_in.
 *   k_out      host; number of distinct pairs (colours after the round).
 * Errors: WL_EINVAL (bad sizes, NULL pointers, k_in > n, or a colour >= k_in
 * when it is detected on the device), WL_EBUDGET, WL_EHIP. */
int wl_refine_round(const wl_csr *g, const uint32_t *color_in, uint32_t k_in,
                    uint64_t seed, uint32_t round, uint32_t *color_out,
                    uint32_t *k_out, void *workspace, uint64_t ws_bytes,
                    void *stream);

/* Algorithm 1 to completion: the coarsest stable colouring refining the
 * initial partition (Theorem 1; with probability >= 1 - rounds * n / p).
 *   g           device CSR.
 *   init_color  device, n labels, or NULL for the trivial partition.  The
 *               initial colour of node i is the dense rank of its label.
 *   max_rounds  cap on rounds (0 = n + 1, which is never reached).
 *   color_out   device, n entries: final colours, dense in [0, k).  These
 *               are the raw lexicographic-rank ids of the last round.
 *   k_out, rounds_out  host; colour count and number of rounds (the
 *               confirming round included; 0 when n == 0).
 * On WL_EMAXROUNDS color_out/k_out/rounds_out hold the state after the last
 * round that ran.  Errors: WL_EINVAL, WL_EBUDGET, WL_EMAXROUNDS, WL_EHIP. */
int wl_stable_coloring(const wl_csr *g, const uint32_t *init_color,
                       uint64_t seed, uint32_t max_rounds, uint32_t *color_out,
                       uint32_t *k_out, uint32_t *rounds_out, void *workspace,
                       uint64_t ws_bytes, void *stream);

/* Allocation-free variant of wl_stable_coloring, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It computes exactly what
 * wl_stable_coloring computes (same colours, colour count and rounds, the
 * same errors) but takes no workspace: its device scratch is a fixed array
 * of WL_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held from
 * the library's load until the process ends.  It calls no hipMalloc,
 * hipFree or other allocating routine, and creates no stream, event or
 * graph (WL_GRAPH and the wl_stats diagnostics do not apply to it).
 *   g, init_color, seed, max_rounds, color_out, k_out, rounds_out
 *               as for wl_stable_coloring (device CSR, device arrays).
 *   stream      must belong to the current device (WL_EINVAL otherwise).
 * Limit: graphs whose wl_workspace_size() without WL_CSR_SYMMETRIC exceeds
 * WL_NOALLOC_SCRATCH_BYTES (about 130 bytes per node plus a few per entry,
 * so some 400,000 nodes) are refused with WL_EBUDGET before any device work.
 * Every call on one GPU uses that GPU's one scratch array: calls that
 * overlap on a GPU (from several threads or streams) race and must be
 * serialised by the caller.  The array keeps the last call's contents;
 * each call initialises all of it that it reads. */
#define WL_NOALLOC_SCRATCH_BYTES (64ull << 20)
int wl_stable_coloring_noalloc(const wl_csr *g, const uint32_t *init_color,
                               uint64_t seed, uint32_t max_rounds,
                               uint32_t *color_out, uint32_t *k_out,
                               uint32_t *rounds_out, void *stream);

/* Algorithm 1 (Section 4.1) for a graph whose edge arrays stay in host
 * memory.  Each round, the rows whose image is needed (those of colour
 * classes with two or more members) are packed by host threads into
 * page-locked staging buffers and copied to the device in chunks of at most
 * 64M entries, on a copy stream of the library's own, while the device
 * computes the images of the previous chunk; the colours, images and the
 * relabel stay in the workspace.  The rounds, seeds and colour ids are those
 * of wl_stable_coloring: for the same graph, labels and seed both return
 * the same colours, colour count and round count.
 *   g_host      host CSR (pageable or page-locked), n < 2^31.
 *   init_host   host labels or NULL (trivial partition).
 *   color_out_host  host, n entries: raw rank ids as from wl_stable_coloring.
 *   workspace   device, 256-byte aligned.  wl_streamed_workspace_size()
 *               gives the size with full chunks (about 69 bytes per node
 *               plus two chunks); a smaller one, down to chunks of 4096
 *               entries, is accepted.  Room beyond that size is used too:
 *               once all chunks of a round fit there, they are kept and the
 *               later rounds need no transfers.  Its contents are scratch.
 * The call also allocates about 2 x 13 bytes (17 weighted) per chunk entry
 * of page-locked host memory, and up to about 25 bytes per node of pageable
 * host memory (the rows a round needs and their segment offsets), freed on
 * return.
 * Errors: WL_EINVAL, WL_EBUDGET, WL_EOVERFLOW, WL_EMAXROUNDS, WL_ENOMEM,
 * WL_EHIP. */
int wl_streamed_workspace_size(const wl_csr *g, uint64_t *bytes_out);
int wl_stable_coloring_streamed(const wl_csr *g_host, const uint32_t *init_host,
                                uint64_t seed, uint32_t max_rounds,
                                uint32_t *color_out_host, uint32_t *k_out,
                                uint32_t *rounds_out, void *workspace,
                                uint64_t ws_bytes, void *stream);

/* Arithmetic of the image z = A w for the calls that this thread makes
 * after it (wl_refine_round, wl_stable_coloring, wl_stable_coloring_streamed,
 * wl_stable_coloring_batched).  q is the precision parameter of Algorithm 1
 * (Section 4.1):
 *   WL_PRECISION_FP (0, the default): the prime field F_p, p = 2^61 - 1.
 *   WL_PRECISION_RING64 (64): the ring R = Z/2^64, as in the paper: values,
 *     sums and products wrap at 2^64.  The k values of a round are pairwise
 *     distinct by construction (distinct stream positions of a bijective
 *     output function), so Algorithm 1's resampling until |H| distinct values
 *     never draws again.  Theorem 1 holds for n <= 2^32 and row sums at most
 *     2^32: the calls check the row sums (on the device for device graphs,
 *     one pass over the weights or row pointers; on the host for host
 *     graphs) and return WL_EOVERFLOW above the bound.
 * In both, node i's new colour is the rank of (c_i, z_i).  Both return the
 * coarsest stable colouring with high probability (Theorem 1), so their
 * partitions agree; the raw colour ids (ranks of different z) differ.
 * wl_set_precision returns WL_EINVAL for another q; wl_get_precision gives
 * the current one. */
#define WL_PRECISION_FP 0u
#define WL_PRECISION_RING64 64u
int wl_set_precision(uint32_t q);
int wl_get_precision(uint32_t *q);

/* Options of wl_stable_coloring_batched.
 * WL_BATCHED_EXACT: when the contraction stops with several batches (the
 *   fixed point of Algorithm 2, or WL_BATCHED_EARLY_STOP), finish with
 *   Algorithm 1 on the last graph (the streamed rounds of
 *   wl_stable_coloring_streamed, from the labels that graph's nodes carry).
 *   A quotient keeps every stable colouring of the graph it contracts
 *   (Definition "Quotient Graph"), so the lifted result is the coarsest
 *   stable colouring refining the labels, as in-core; coarsest_out is 1.
 * WL_BATCHED_EARLY_STOP: the termination used in Section 5.4: stop the
 *   outer loop as soon as the next iteration would not have fewer batches. */
#define WL_BATCHED_EXACT 1u
#define WL_BATCHED_EARLY_STOP 2u

/* Algorithm 2 (Section 4.2) for graphs whose edge arrays stay in host
 * memory; only one batch of entries is on the device at a time.  Each batch
 * runs Algorithm 1 with the nodes outside it frozen as singletons; the
 * quotient graphs between outer iterations are built on the device, chunk by
 * chunk, and kept in pageable host memory that this call allocates and frees
 * (at most 8 bytes per entry of the input, plus 8 bytes per node, for each
 * of the two quotients alive at a time).  Needs n < 2^30.
 *   g_host      host CSR, pageable or page-locked.  Page-locked arrays are
 *               copied to the device by DMA directly; pageable ones (and the
 *               library's quotients) through page-locked staging buffers of
 *               64 MiB that the call allocates (two per copy stream: the
 *               quotient's copies in and out run on two host threads and
 *               streams of their own, overlapped with the device's work;
 *               without page-locked memory the copies go unstaged).
 *   init_host   host labels or NULL (trivial partition).
 *   max_batch_entries  cap M_b on entries per batch; 0 = the largest cap the
 *               workspace allows.  Batches are contiguous CSR entry ranges
 *               cut at row boundaries; a row longer than the cap is split and
 *               its node is a boundary node.
 *   color_out_host  host, n entries: first-occurrence canonical colours
 *               (node 0 gets 0, each new colour the next id), so equal
 *               partitions give equal arrays.
 *   options     0, or WL_BATCHED_EXACT and / or WL_BATCHED_EARLY_STOP.
 *   k_out, rounds_out (sum over all batch runs and the exact finish),
 *   outer_out (outer iterations), coarsest_out (1 when the last outer
 *   iteration had a single batch or the exact finish ran, which makes the
 *   result the coarsest stable colouring; 0 when the contraction stopped
 *   with several batches).
 * The exact finish needs the workspace of wl_stable_coloring_streamed for
 * the graph it runs on, at least with chunks of 4096 entries.
 * WL_BATCHED_EXACT is accepted only for graphs of at most 2^31 entries, the
 * largest on which the exact finish has been verified (WL_EINVAL above;
 * one run on a 1.7e10-entry graph ended in a host fault whose cause has not
 * been found).  wl_stable_coloring_streamed computes the same colouring
 * (the coarsest stable one) for larger graphs.
 * Errors: WL_EINVAL (also unknown option bits), WL_EBUDGET, WL_EOVERFLOW,
 * WL_EMAXROUNDS, WL_ENOMEM, WL_EHIP. */
int wl_stable_coloring_batched(const wl_csr *g_host, const uint32_t *init_host,
                               uint64_t seed, uint64_t max_batch_entries,
                               uint32_t options, uint32_t *color_out_host,
                               uint32_t *k_out, uint32_t *rounds_out,
                               uint32_t *outer_out,
                               int *coarsest_out, void *workspace,
                               uint64_t ws_bytes, void *stream);

/* Exact stability certificate (Definition "Stable Coloring", Section 3):
 * WL_OK when every two nodes of each colour class have equal total
 * out-weight into every class, WL_ENOTSTABLE otherwise.  Deterministic (no
 * randomness).  An entry of weight 0 adds nothing to a total, so it is the
 * same as a missing entry.  Applied to the output of Algorithm 1 it turns
 * the probabilistic guarantee of Theorem 1 into a certainty: every colouring
 * Algorithm 1 produces is at least as coarse as the coarsest stable colouring
 * refining its start, so one that passes this check is exactly that one.
 *   g          device CSR.
 *   color      device, n entries, each < k (ids need not all be used).
 *   k          1 <= k <= n (any k when n == 0).
 *   workspace  device, 256-byte aligned, >= wl_verify_workspace_size(g)
 *              bytes (4 bytes per entry, 8 for weighted graphs, plus about
 *              17 bytes per node); its contents are scratch.
 * Errors: WL_EINVAL (NULL pointers, k out of range, a colour >= k), WL_EBUDGET,
 * WL_EHIP. */
int wl_verify_workspace_size(const wl_csr *g, uint64_t *bytes_out);
int wl_verify_stable(const wl_csr *g, const uint32_t *color, uint32_t k,
                     void *workspace, uint64_t ws_bytes, void *stream);

/* Message for the last non-zero return on this thread ("" if none). */
const char *wl_last_error(void);

/* Diagnostics (instrumentation of this library, not part of the method).
 * wl_stats_enable(flags) turns them on for the calling thread:
 *   WL_STATS_TIME  record HIP events on 'stream' around every image launch
 *                  (step "z = A w" of a round) and around the whole call;
 *   WL_STATS_WORK  also count, with one extra reduction kernel per round,
 *                  the rows and CSR entries each image launch reads (this
 *                  adds device work: use it in an untimed run).
 * The image of a round is one of three kinds: 'gather' (a row reads its
 * neighbours' values), 'pb' (propagation blocking on a symmetric graph: its
 * passes count as one launch) or 'uniform' (rounds with a single colour).
 * With WL_GRAPH=1 in the environment, the rounds that run without a
 * read-back are replayed from a HIP graph: their image launches are counted
 * but not timed, so 'ms' then covers the host-driven rounds only.
 * wl_stats_get() returns the figures of the last in-core call on this thread.
 * Both return WL_OK, or WL_EINVAL for a NULL pointer / unknown flag. */
#define WL_STATS_TIME 1
#define WL_STATS_WORK 2
typedef struct wl_stats_kind {
    uint32_t launches;         /* image launches of this kind               */
    uint32_t pad;
    double ms;                 /* their summed device time (WL_STATS_TIME)  */
    uint64_t rows;             /* rows whose image they computed (WORK)     */
    uint64_t entries;          /* CSR entries they read (WORK)              */
} wl_stats_kind;
typedef struct wl_stats {
    uint32_t rounds;           /* rounds of the last call                   */
    uint32_t pad;
    double call_ms;            /* device time of the whole call             */
    wl_stats_kind gather;
    wl_stats_kind pb;
    wl_stats_kind uniform;
} wl_stats;
int wl_stats_enable(int flags);
int wl_stats_get(wl_stats *out);

/* Environment variables read by the library (tuning and diagnostics; none
 * changes a result):
 *   WL_VALIDATE=1        device checks of the graph (see the conventions).
 *   WL_PB=0 | force      propagation blocking off, or on whenever possible
 *                        (default: on when at least half the entries feed
 *                        rows whose image is needed).
 *   WL_DEGREE_ROUND=0    no histogram round from one colour.
 *   WL_HOST_ROUNDS=n     rounds driven from the host before the device-driven
 *                        ones (default 8).
 *   WL_ASYNC_PASSES=n    radix passes a device-driven round launches (0-8).
 *   WL_GRAPH=1           replay the device-driven rounds from a HIP graph.
 *   WL_NT_STREAM=1       non-temporal loads of the column indices.
 *   WL_SORT_FIX=n        largest mixed bucket the counting sorts of the
 *                        segments of 65 to 2048 nodes fix by insertion
 *                        (default 32; 0 sends every segment with one to the
 *                        sorting networks).
 *   WL_CHAIN_SPINS=n     polls a chained scan of the incremental rounds
 *                        waits for an earlier chunk before it gives up
 *                        (default and maximum 2^22, far beyond any real
 *                        wait).  A test hook: with a tiny bound a call
 *                        either completes with the same result or fails
 *                        with WL_EHIP ("a chained scan did not complete"),
 *                        never returns a different result.
 *   WL_HOST_STAGING=0    copy pageable host memory without page-locked
 *                        staging buffers (as when they are refused).
 *   WL_TRACE_STREAMED=1, WL_TRACE_BATCHED=1
 *                        per-round (per outer iteration) host-side timings
 *                        of the streamed rounds (of Algorithm 2) on stderr. */

#ifdef __cplusplus
}
#endif

#endif /* WL_H */
