/*
 * massive.h - C ABI of libmassive: one graph partition's per-minibatch
 * sampling + halo prefetch buffer + feature gather, after MassiveGNN
 * (Sarkar, Ghosh, Tallent, Jannesari, arXiv 2410.22697), on one MI355X.
 *
 * The three calls follow the paper's procedures:
 *   massive_init        INITIALIZE_PREFETCHER (Algorithm 1)
 *   massive_sample      PREFETCH_WITH_EVICTION up to the eviction check
 *                       (Algorithm 2: NeighborSampler, hit/miss split, S_E
 *                       decay, local/buffer copies, miss fetch, S_A update)
 *   massive_evict_step  the periodic round of Algorithm 2 (EVICT_AND_REPLACE
 *                       with the score swap of Section IV-B, threshold Eq. 1)
 *
 * Ids. The partition's nodes carry partition-local ids: local (owned)
 * nodes [0, L), halo (remote) nodes [L, L+H). The prefetcher's state and the
 * eviction outputs use halo indices h = id - L in [0, H).
 *
 * Semantics (readings of the paper, fixed so that results are exact):
 *   - The sampler walks G_p, the CSR of the subgraph induced on local + halo
 *     nodes. Fanouts are hop-first. Hop k (1-based) samples for every node
 *     of frontier F_{k-1}; new nodes are appended in ascending id, so F_k is
 *     a prefix of F_{k+1} and the seeds come first.
 *   - For a row v of length d at global step t, hop k: if d <= fanout every
 *     position is kept; otherwise the fanout positions j with the smallest
 *     (key_j, j), where key_j is word (j mod 4) of Philox4x32-10 (Salmon et
 *     al., SC'11) with counter (j/4, v, t, k) and key (seed_lo, seed_hi).
 *     Sampled neighbours are emitted in ascending j.
 *   - Halo rank orders halo nodes by (degree desc, global id asc); the
 *     buffer starts with the cap = floor(H * buffer_pct / 100) best ranked.
 *   - Hits/misses use the buffer as it stood at the start of the step.
 *     Every step: S_E *= gamma (fp32, one product per step) for each
 *     buffered node not sampled; S_A += 1 for each miss.
 *   - t counts steps across epochs from 0. After step t, if t > 0 and
 *     t mod delta == 0, the round evicts the slots with S_E < alpha, where
 *     alpha is gamma multiplied delta times in fp32, and replaces them with
 *     the unbuffered halo nodes of highest (S_A, then rank); evicted slots
 *     in ascending order are paired with replacements in that order. If
 *     there are fewer candidates k' than evictions, the k' slots with the
 *     smallest (S_E, rank) are evicted. Swap: evicted node's S_A := its last
 *     S_E, slot's S_E := the replacement's last S_A, replacement's S_A := -1.
 *
 * Threading: calls on one context must not overlap. Different contexts are
 * independent. A context in MASSIVE_LINK_STAGED mode runs host threads of
 * its own, which end in massive_destroy. Every call returns a status;
 * nothing throws across the ABI.
 */
#ifndef MASSIVE_H
#define MASSIVE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define MASSIVE_OK 0
#define MASSIVE_EINVAL (-1)    /* bad argument (message in massive_last_error) */
#define MASSIVE_ECAPACITY (-2) /* an output buffer is smaller than the bound  */
#define MASSIVE_ENOMEM (-3)    /* device or host allocation failed            */
#define MASSIVE_EHIP (-4)      /* HIP runtime error; from a step or a round, the
                                  context then takes no further work         */
#define MASSIVE_ESTATE (-5)    /* call out of order (see massive_sample)      */

#define MASSIVE_MAX_HOPS 8

/* S_A layouts (massive_init_args.score_layout), the two the paper weighs in
 * Section IV-B: an array over the halo only, or one over every global id */
#define MASSIVE_SCORES_BY_RANK 0 /* S_A over the H halo nodes, in rank order */
#define MASSIVE_SCORES_BY_GID 1  /* S_A over all n_global global ids, indexed by id */
#define MASSIVE_MAX_INFLIGHT 3 /* batches enqueued and not yet waited for */

/* How rows cross the host link (massive_init_args.link_mode): the misses,
 * hits on slots still refilling, and the replacement rows of Algorithm 2's
 * merged fetch. Both modes give the same results. */
#define MASSIVE_LINK_LOADS 0  /* kernels read the mapped pinned store */
#define MASSIVE_LINK_STAGED 1 /* host threads gather the rows into pinned
                                 staging memory, the DMA engines copy them to
                                 the device and a kernel scatters them; no
                                 kernel reads host memory, so kernels running
                                 beside the path (a trainer) are not slowed */

typedef struct massive_ctx massive_ctx;

/* Inputs of massive_init. Every host array is read during the call only,
 * except halo_store, which the context borrows until massive_destroy. */
typedef struct {
  int32_t L;                  /* local nodes, ids [0, L)                      */
  int32_t H;                  /* halo nodes, ids [L, L+H)                      */
  const int64_t* indptr;      /* host [L+H+1], G_p row offsets (int64)        */
  const int32_t* indices;     /* host [indptr[L+H]], partition-local ids      */
  const int32_t* halo_gid;    /* host [H], global id of halo h (rank ties)    */
  const int64_t* halo_degree; /* host [H], degree used to rank halo nodes     */
  const void* local_feat;     /* host [L * row_bytes], copied into HBM        */
  const void* halo_store;     /* PINNED host [H * row_bytes] (hipHostMalloc'd,
                                 e.g. a torch pin_memory tensor): the remote
                                 features; read by the GPU over the host link */
  int64_t row_bytes;          /* bytes per feature row, multiple of 4, <= 1 MiB */
  int32_t K;                  /* hops, 1..MASSIVE_MAX_HOPS                     */
  int32_t fanout[MASSIVE_MAX_HOPS]; /* hop-first fanouts, each >= 1           */
  int32_t buffer_pct;         /* f_p^h as an integer percent, 0..100          */
  float gamma;                /* decay factor, 0 < gamma <= 1                 */
  int32_t delta;              /* eviction interval, >= 1                      */
  uint64_t seed;              /* Philox key                                   */
  void* stream;               /* hipStream_t for all work (NULL: default)     */
  int32_t score_layout;       /* MASSIVE_SCORES_BY_RANK (0, the default) or
                                 MASSIVE_SCORES_BY_GID: S_A (and a rank per
                                 id) over every global id, 8 B per id; the
                                 eviction round then selects over all ids  */
  int64_t n_global;           /* MASSIVE_SCORES_BY_GID: the global id space,
                                 every halo_gid in [0, n_global) and distinct,
                                 n_global <= 2^31; ignored otherwise         */
  int32_t link_mode;          /* MASSIVE_LINK_LOADS (0, the default) or
                                 MASSIVE_LINK_STAGED                          */
  int32_t link_threads;       /* MASSIVE_LINK_STAGED: host threads gathering
                                 rows, 1..64 (0: 8); the context starts them
                                 and one more that feeds the copies          */
} massive_init_args;

/* Creates a context: uploads G_p and local features to HBM, ranks the halo,
 * fills the HBM buffer with the cap best-ranked halo rows from halo_store,
 * and sets S_E = 1, S_A = -1 / 0. Both score layouts give the same results
 * (states, eviction and replacement sets); they differ in memory and in the
 * eviction round's time. MASSIVE_EINVAL for a halo_gid outside [0, n_global)
 * or repeated (BY_GID). On failure *out is NULL and the message is in
 * massive_last_error(NULL). */
int massive_init(const massive_init_args* args, massive_ctx** out);

/* Upper bounds on the output sizes of a batch of n_seeds seeds:
 * n_bound[0..K] frontier sizes, e_bound[0..K-1] sampled edges per hop. */
int massive_output_bounds(const massive_ctx* ctx, int32_t n_seeds, int64_t* n_bound,
                          int64_t* e_bound);

/* Caller-owned device buffers of one batch, plus the sizes written back.
 * Capacities are in elements; each must be at least the bound above. */
typedef struct {
  int32_t* nodes;                          /* [nodes_cap] F_K; F_k = nodes[0:n[k]] */
  uint8_t* mask;                           /* [nodes_cap] 0 local, 1 hit, 2 miss   */
  void* feat;                              /* [nodes_cap * row_bytes], row i is the
                                              feature row of nodes[i]             */
  int64_t nodes_cap;
  /* entry k (0-based) is the block of hop k+1, which samples for the n[k]
   * rows of F_k: indptr[k] has n[k]+1 offsets into indices[k], and
   * indices[k] holds e[k] sampled neighbours as positions in nodes */
  int32_t* indptr[MASSIVE_MAX_HOPS];
  int32_t* indices[MASSIVE_MAX_HOPS];
  int64_t indptr_cap[MASSIVE_MAX_HOPS];
  int64_t indices_cap[MASSIVE_MAX_HOPS];
  /* written by massive_sample */
  int64_t n[MASSIVE_MAX_HOPS + 1];         /* frontier sizes n_0..n_K              */
  int64_t e[MASSIVE_MAX_HOPS];             /* sampled edges per hop                */
  int64_t local, hits, misses;             /* input rows by class (unique nodes)   */
  int64_t host_rows;                       /* rows read over the host link: the
                                              misses, plus hits on slots whose
                                              refill had not landed yet        */
} massive_batch;

/* One minibatch at the context's current step t: samples K hops from the
 * n_seeds device seeds (distinct local ids), classifies every frontier node
 * against the buffer, updates the scores and gathers all feature rows (HBM
 * rows from the local slab and the buffer, misses from halo_store). Returns
 * after the batch is complete on the device (massive_sample_async followed by
 * massive_batch_wait); t advances by one.
 * MASSIVE_ESTATE if the previous step's massive_evict_step was not called.
 * MASSIVE_EINVAL (no state change) if a seed is out of [0, L) or repeated. */
int massive_sample(massive_ctx* ctx, const int32_t* seeds, int32_t n_seeds, massive_batch* io);

/* massive_sample for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same step and the same results, but its per-step scratch (sizes, gather
 * lists, scan flags) lives in one static device array per GPU, of fixed size,
 * instead of the context's per-slot buffers, and the call itself allocates
 * nothing (no hipMalloc, no event creation; timing is off for it). Limit:
 * frontier bound n_bound[K] <= 1,310,720 rows; a larger bound is refused with
 * MASSIVE_ECAPACITY. Synchronous, and refused (MASSIVE_ESTATE) while a batch
 * of this context is in flight. Calls that overlap on one GPU, from any
 * contexts, race on that array: serialise them. */
int massive_sample_noalloc(massive_ctx* ctx, const int32_t* seeds, int32_t n_seeds, massive_batch* io);

/* The asynchronous form of massive_sample, for look-ahead (Algorithm 1
 * prepares the next minibatch while the current one is consumed): enqueues
 * the step and returns at once. The batch's buffers must not be read or
 * reused, and its sizes are not written, until massive_batch_wait returns for
 * it. At most MASSIVE_MAX_INFLIGHT batches are in flight: the next steps can
 * be enqueued (each after its predecessor's massive_evict_step) while earlier
 * ones still read misses over the host link; a further one is refused with
 * MASSIVE_ESTATE. Argument errors are returned here; seed errors
 * are returned by massive_batch_wait (if a later step was already issued the
 * context then refuses further work with MASSIVE_ESTATE). */
int massive_sample_async(massive_ctx* ctx, const int32_t* seeds, int32_t n_seeds, massive_batch* io);

/* Waits for the batch enqueued with io and writes its sizes and counters.
 * MASSIVE_EINVAL for a seed out of [0, L) or repeated (the step is taken
 * back if no later step was issued); MASSIVE_EHIP, and the context refuses
 * further work, if the sampler's threshold search found no acceptable
 * candidate count or a single-pass scan waited past its bound (neither is
 * expected), or if an eviction round produced inconsistent indices.
 * MASSIVE_ESTATE for a batch issued after a step that failed in any of these
 * ways (whichever of the two is waited for first): it was sampled against the
 * failed step's leftover state, so its outputs are not valid. */
int massive_batch_wait(massive_ctx* ctx, massive_batch* io);

/* The eviction round owed by the step just sampled; must be called once after
 * every massive_sample / massive_sample_async. Runs the round iff that step t
 * has t > 0 and t mod delta == 0. The round is decided on the device, on the
 * library's copy stream, beside the next step's sampling (that step's lookup
 * waits for it): with k_out == NULL the call only enqueues it; otherwise it
 * waits for the round and writes k' (0 when no round is due). Optional device
 * outputs, each with room for cap entries: evicted halo ids, the slots they
 * held (ascending), and their replacements (entries [0, k')); they are
 * complete when the call returns with k_out, or once the next step's
 * massive_batch_wait has returned. The replacement rows are copied from
 * halo_store on the copy stream; until they have landed, the next steps read
 * hits on those slots from halo_store (the same bytes) and write them into
 * their slots, so that no row crosses the host link twice. */
int massive_evict_step(massive_ctx* ctx, int32_t* evicted, int32_t* slots, int32_t* replaced,
                       int64_t* k_out);

/* Totals since init (each pointer may be NULL): rounds that evicted at least
 * one slot, slots evicted, and rows the refill copied over the host link
 * (including the initial fill of the buffer; a replacement whose row a miss
 * gather already wrote into its slot is not copied again). Waits for the
 * refill chunks launched so far. */
int massive_get_counters(massive_ctx* ctx, int64_t* rounds, int64_t* evicted, int64_t* refilled);

/* Host copies of the prefetcher state (each pointer may be NULL):
 * slot_id[cap] halo id per slot, S_E[cap], S_A[H], steps sampled so far. */
int massive_get_state(massive_ctx* ctx, int32_t* slot_id, float* S_E, float* S_A, int64_t* t);

/* Host copy of the HBM buffer's rows, [cap * row_bytes]. */
int massive_get_buffer_rows(massive_ctx* ctx, void* host_out);

/* cap (buffer slots) and alpha (each pointer may be NULL). */
int massive_info(const massive_ctx* ctx, int64_t* cap, float* alpha);

/* Per-kernel-group timing with HIP events recorded on the stream each group
 * runs on (the groups of massive_get_timing). groups is a bit mask, bit i for
 * group i (MASSIVE_TIMING_ALL: every group, 0: off); it clears the totals.
 * Each timed group adds event packets to its streams, so a run that must not
 * be slowed times only what it needs. MASSIVE_EINVAL for bits outside the
 * mask. */
#define MASSIVE_TIMING_ALL 0x7F
int massive_set_timing(massive_ctx* ctx, int groups);
/* Totals since enabled: out_ms[i] summed milliseconds and out_calls[i]
 * launches for i = 0 sample+dedup, 1 classify, 2 gather_hbm, 3 gather_miss,
 * 4 eviction round, 5 refill, 6 the last hop's sampler kernel alone (a part
 * of group 0). out_ms and out_calls have room for 7 entries each.
 * Synchronises the context's streams. */
int massive_get_timing(massive_ctx* ctx, double* out_ms, int64_t* out_calls);

/* Frees every device and host resource of the context; NULL is a no-op.
 * Always MASSIVE_OK. */
int massive_destroy(massive_ctx* ctx);

/* Message of the last failure on this context (ctx == NULL: of the last
 * failed massive_init on this thread). Never NULL. */
const char* massive_last_error(const massive_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* MASSIVE_H */
