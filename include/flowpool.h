/*
 * flowpool.h -- C ABI of libflowpool: the consumer side of a unified memory
 * pool for decoupled VLM training, on one MI355X (gfx950).
 *
 * Producers (frozen vision encoders) write each sample's vision embeddings
 * into pages of the pool, together with the sample's text token ids and the
 * metadata that pairs them (paper Sec. 3.1 workflow; Sec. 3.2, producer
 * side). A planner groups resident samples into cost-balanced microbatches
 * (Sec. 3.4, Eq. 3). The backbone consumes a microbatch by sample id: the
 * library resolves every visual row's GVA through the page table, gathers the
 * page rows and the text-embedding-table rows and packs them into one varlen
 * microbatch with cu_seqlens and position ids (Sec. 3.1: consumers address
 * data by GVA only; Sec. 3.2: translation through locally held page tables).
 *
 * Conventions for every entry point:
 *  - Return value: FP_OK (0) or a negative FP_E* status. Nothing throws or
 *    aborts across the ABI. fp_last_error() returns a message for the last
 *    failing call on the calling thread.
 *  - A failing call leaves the pool unchanged and launches nothing. Host
 *    memory exhausted inside a call returns ENOMEM (the one case where a
 *    call that already changed the pool may not have undone it).
 *  - "host" pointers are ordinary CPU memory read or written before the call
 *    returns; "device" pointers must be readable/writable by the GPU (device
 *    memory, or pinned host memory mapped into the GPU address space).
 *  - `stream` is a hipStream_t cast to void* (NULL = the null stream). Work
 *    is enqueued on it. The pool orders its own work across streams: a pack
 *    or plan of a sample waits (on the GPU) for the sample's write if that
 *    was enqueued on another stream and has not finished, and a free of a
 *    sample still being read by an enqueued pack is deferred until that
 *    pack completes (Sec. 3.1: producers and consumers run decoupled).
 *    For that, the pool remembers the streams that packed each sample: a
 *    stream passed to pack_microbatch (or pool_write_sample) must stay valid
 *    until the samples it packed are freed, the pool is destroyed, or the
 *    caller has handed it to pool_forget_stream.
 *  - Embeddings are bf16, row-major, H elements per row; the library moves
 *    them as raw 16-bit words (NaN payloads, signed zeros and denormals are
 *    preserved exactly).
 *  - Calls from several threads are serialised internally by a mutex, so a
 *    producer thread and a consumer thread may share one pool.
 *  - HIP graphs: pack_microbatch may be captured on a capturing stream when
 *    its row table travels in the kernel arguments (at most 32 samples whose
 *    rows form at most 160 runs, a run being a stretch of one sample's text
 *    rows, or of its image rows with no text row between them) and its
 *    samples' writes are known complete (a pack, plan or pool_reclaim after they finished has seen
 *    them; the capture makes no event queries); each replay packs the same
 *    samples into the same buffers, through the page lists they had at
 *    capture. A captured pack therefore holds its samples: pool_free_sample
 *    and pool_migrate return ESTATE for them until the caller, once the
 *    graph will not be replayed again, hands the same sample id list to
 *    pool_release_captured (once per captured pack). pool_write_sample,
 *    pool_migrate and plan_microbatches return ESTATE on a capturing stream,
 *    as does a pack that cannot be captured.
 */
#ifndef FLOWPOOL_H
#define FLOWPOOL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FP_ABI_VERSION 5

typedef struct fp_pool fp_pool;   /* opaque; created and owned by the library */
typedef int32_t fp_status;

enum {
  FP_OK = 0,
  FP_EINVAL = -1,     /* bad argument (value, size, id, position, policy) */
  FP_ENOMEM = -2,     /* pool pages, sample slots or metadata arena exhausted */
  FP_ENOENT = -3,     /* unknown or already-freed sample id */
  FP_ECAPACITY = -4,  /* microbatch rows exceed the output capacity */
  FP_EALIGN = -5,     /* pointer not aligned as required */
  FP_EHIP = -6,       /* a HIP runtime call failed (message names it) */
  FP_ESTATE = -7      /* call not valid in the pool's state */
};

enum { FP_ALLOC_CONTIG = 0, FP_ALLOC_SCATTER = 1 };
enum { FP_TIER_HBM = 0, FP_TIER_HOST = 1 };
enum { FP_TIER_MASK_HBM = 1, FP_TIER_MASK_HOST = 2, FP_TIER_MASK_ALL = 3 };

/* Pool configuration (Sec. 3.2).
 *  hidden        H, bf16 elements per row; 2*H must be a multiple of 16.
 *  page_tokens   P, rows per page; page bytes pb = P * 2H.
 *  hbm_pages     pages backed by device memory (HBM tier).
 *  host_pages    pages backed by pinned host memory that kernels read over
 *                PCIe (DRAM tier); 0 = untiered.
 *  alloc_policy  FP_ALLOC_CONTIG: a sample's pages are the lowest-index run
 *                of consecutive free pages in one tier (HBM tried first).
 *                FP_ALLOC_SCATTER: pages are popped one at a time from a
 *                per-tier LIFO free stack (page 0 first on a fresh pool);
 *                a freed sample's pages are pushed last-page-first.
 *  device        HIP device ordinal the pool lives on.
 *  vocab         text ids must lie in [0, vocab); 0 = samples carry no text.
 *  gva_start     base of the GVA space, a multiple of 4096; 0 = 0x100000000000.
 *                The HBM region is [gva_start, gva_start + world_size*hbm_pages*pb),
 *                the DRAM region follows it; this rank owns
 *                [region + rank*max_size, region + (rank+1)*max_size) of each.
 *  world_size, rank   must be 1 and 0 in this library (single process).
 *  max_samples   resident sample slots; 0 = 65536.
 *  meta_bytes    device metadata arena (text ids, image positions, page
 *                lists); 0 = 64 MiB, at most 8 GiB.
 *  frame_shuffle_seed  0 = physical frames bound to GVA pages in order; else
 *                a seeded permutation of frames (placement-independence tests).
 *  chunk_bytes   the library allocates tier backing in chunks of this many
 *                bytes (rounded down to whole pages); 0 = 1 GiB.
 *  hbm_backing   NULL = the library allocates the HBM tier's backing;
 *                else caller-owned device memory of `device`, 256-byte
 *                aligned, with at least hbm_pages * 2H * page_tokens bytes
 *                from this address inside one allocation (e.g. a torch
 *                tensor). The pool binds its frames to it in order and never
 *                frees it; it must stay valid until pool_destroy.
 *  host_backing  the same for the host tier: caller-owned pinned host memory
 *                mapped into the GPU at the same address (hipHostMalloc, a
 *                torch pinned tensor), host_pages * 2H * page_tokens bytes.
 *  pack_cus      compute units the pack's chunk geometry is sized for (the
 *                chunks of its last wave and a half of resident workgroups are
 *                8 KiB, then 4 KiB); 0 = the device's count. It changes timing
 *                only, never results; tests set it small to reach every chunk
 *                size.
 *  reserved      must be 0.
 */
typedef struct fp_pool_config {
  int32_t hidden;
  int32_t page_tokens;
  int64_t hbm_pages;
  int64_t host_pages;
  int32_t alloc_policy;
  int32_t device;
  int64_t vocab;
  uint64_t gva_start;
  int32_t world_size;
  int32_t rank;
  int64_t max_samples;
  int64_t meta_bytes;
  uint64_t frame_shuffle_seed;
  int64_t chunk_bytes;
  void* hbm_backing;
  void* host_backing;
  int32_t pack_cus;
  int32_t reserved;
} fp_pool_config;

/* Library ABI version (FP_ABI_VERSION of the build). */
int32_t fp_abi_version(void);

/* Message for the last non-OK status returned on this thread ("" if none).
 * The string is owned by the library and valid until the next call. */
const char* fp_last_error(void);

/* Fill *cfg with defaults (all zero except world_size = 1). */
void fp_config_init(fp_pool_config* cfg);

/* Create a pool (Sec. 3.2 initialisation): reserve this rank's GVA segments,
 * allocate the tiers' physical memory, bind it to the GVA pages through the
 * page table and upload the table to the device. cfg: host. *out receives the
 * pool handle. Errors: EINVAL (bad field; a backing of the wrong kind, device
 * or size), EALIGN (a backing not 256-byte aligned), EHIP (allocation
 * failed). */
fp_status pool_create(const fp_pool_config* cfg, fp_pool** out);

/* Destroy a pool and free all its memory (the library's; the paper describes
 * no teardown). The caller must have synchronised every stream that still
 * uses it. NULL is accepted. */
fp_status pool_destroy(fp_pool* p);

/* Producer write (Sec. 3.2: each producer writes vision embeddings and text
 * tokens into its own process's GVA segment; Sec. 3.1 pairing metadata).
 *  text_ids        host int32[n_text], each in [0, vocab).
 *  img_pos         host int32[n_img], nondecreasing, each in [0, n_text]: image
 *                  j is placed before text token img_pos[j] (after all text
 *                  when equal to n_text); equal positions keep image order.
 *  img_ntok        host int32[n_img] >= 0, visual rows of each image.
 *  vis_emb         device bf16 [sum(img_ntok), H] row-major, images
 *                  concatenated in order, 16-byte aligned; it is read on
 *                  `stream` after the call returns and must stay valid until
 *                  that work completes. NULL reserves the pages without
 *                  writing them (their rows are then unspecified).
 *  page_tier_wish  host uint8[ceil(sum(img_ntok)/P)] of FP_TIER_* per page
 *                  (SCATTER only; a full tier falls back to the other); NULL =
 *                  HBM first.
 * The sample's visual rows fill its own pages densely in order (last page
 * possibly partial). All-or-nothing. *out_sample_id (host) receives a new id,
 * never reused, >= 1.
 * Errors: EINVAL (positions, counts, ids, empty sample, wish, more than
 *         2^31 - 1024 16-byte vectors of visual rows, vis_emb in memory the GPU cannot
 *         read, such as ordinary pageable host memory), EALIGN,
 * ENOMEM (pages, slots or metadata exhausted), EHIP. */
fp_status pool_write_sample(fp_pool* p, const int32_t* text_ids, int32_t n_text,
                            const int32_t* img_pos, const int32_t* img_ntok, int32_t n_img,
                            const void* vis_emb, const uint8_t* page_tier_wish,
                            void* stream, uint64_t* out_sample_id);

/* Release a sample; its id becomes invalid at once. The paper's pool
 * (Sec. 3.2) describes writing and consuming samples but defines no release;
 * this is the library's, so that the pool can be reused over a run. Its
 * pages, metadata and slot return to the free lists as soon as the work
 * enqueued before this call on every stream that packed the sample has
 * completed: at once if those streams are idle, otherwise later (an event
 * recorded on each busy one; event-deferred reclamation, checked by the next
 * write or by pool_reclaim). If the sample's own write has not finished, the
 * call waits for it. Pages freed while no pack is pending return in free
 * order.
 * Errors: ENOENT, ESTATE (a captured pack still holds the sample), EHIP. */
fp_status pool_free_sample(fp_pool* p, uint64_t sample_id);

/* The library's side of pool_free_sample (the paper defines no release):
 * returns the resources of deferred frees whose packs have completed (with
 * wait != 0, first waits for all of them), and forgets the events of writes
 * that have completed (all of them with wait != 0). *out_deferred_pages
 * (host, may be NULL) receives the pages still deferred. pool_write_sample reclaims by
 * itself and, when memory runs short, waits for the packs holding deferred
 * pages. Errors: EHIP. */
fp_status pool_reclaim(fp_pool* p, int32_t wait, int64_t* out_deferred_pages);

/* Tier migration (Sec. 3.2: the pool spans HBM and host DRAM; data moves
 * between tiers by the copy engine the pair of tiers calls for). Moves every
 * page of the samples sample_ids[0..n) that is not in `tier` (FP_TIER_HBM or
 * FP_TIER_HOST) into a free page of `tier`: pages in visual-row order, each
 * taking the next page of the tier's free stack, so a sample's GVAs change
 * and its bytes do not. The copies are asynchronous DMA copies on `stream`
 * (host <-> device through the SDMA engines; device <-> device as a copy),
 * followed by the upload of the samples' new page lists. Packs and plans
 * enqueued later on other streams wait for them; packs enqueued earlier keep
 * reading the old pages, which return to their tier's free stack
 * (last-page-first) once the copies and those packs have completed. Used to
 * prefetch host-tier pages into HBM ahead of their packs, or to demote
 * samples to the host tier. SCATTER pools only; a sample may be listed once.
 * All-or-nothing. *out_pages_moved (host, may be NULL) receives the number of
 * pages moved. Errors: EINVAL, ENOENT, ENOMEM (not enough free pages in
 * `tier`, or metadata arena full), ESTATE (a captured pack holds a listed
 * sample, or `stream` is capturing), EHIP. */
fp_status pool_migrate(fp_pool* p, const uint64_t* sample_ids, int32_t n, int32_t tier,
                       void* stream, int64_t* out_pages_moved);

/* Planning policies. */
enum {
  FP_PLAN_LPT = 0,     /* each sample to the fitting microbatch of least accumulated cost */
  FP_PLAN_ZIGZAG = 1   /* the sample at position p of the order to microbatch snake(p) */
};

/* Planner (Sec. 3.4): evaluate each sample's cost K*l + l^2 (the per-sample
 * cost l + l^2/K scaled by K; l = text + visual rows) with a GPU kernel over
 * the device sample table, then partition into n_mb microbatches of at most
 * `capacity` tokens, samples taken by decreasing cost (ties: lower index):
 *  FP_PLAN_LPT      each to the fitting microbatch of least accumulated cost
 *                   (ties: lower microbatch index);
 *  FP_PLAN_ZIGZAG   the sample at position p of that order to microbatch
 *                   snake(p), snake = 0, 1, ..., n_mb-1, n_mb-1, ..., 0, 0, 1, ...
 *                   (Alg. 1's zig-zag dealing, applied to samples); if it
 *                   has no room, to the first with room among snake(p+1),
 *                   snake(p+2), ...
 * A sample that fits nowhere is deferred (-1) and stays resident. Samples of
 * one microbatch keep their order in sample_ids.
 *  sample_ids       host uint64[n], distinct, resident.
 *  out_assign       host int32[n]: microbatch index or -1.
 *  out_mb_tokens    host int32[n_mb]: tokens per microbatch.
 *  out_mb_cost_scaled  host int64[n_mb]: sum of K*l + l^2 per microbatch.
 *  out_mb_max_len   host int32[n_mb] or NULL: longest sample per microbatch
 *                   (with out_mb_tokens this gives Eq. 3).
 *  out_sample_cost_scaled  host int64[n] or NULL: the per-sample costs.
 * Synchronous: returns after `stream` has finished the cost kernel.
 * Errors: EINVAL (n_mb outside [1, 2^20], capacity < 1, cost_k < 1, policy,
 * duplicates), ENOENT, EHIP. */
fp_status plan_microbatches(fp_pool* p, const uint64_t* sample_ids, int32_t n,
                            int32_t capacity, int32_t n_mb, int32_t cost_k, int32_t policy,
                            int32_t* out_assign, int32_t* out_mb_tokens,
                            int64_t* out_mb_cost_scaled, int32_t* out_mb_max_len,
                            int64_t* out_sample_cost_scaled, void* stream);

/* The partition step of plan_microbatches (Sec. 3.4: samples balanced across
 * microbatches by cost) on given lengths and costs, host only
 * (no pool, no GPU). lengths: host int32[n] >= 1; costs_scaled: host
 * int64[n]; outputs as in plan_microbatches. Errors: EINVAL. */
fp_status plan_partition(const int32_t* lengths, const int64_t* costs_scaled, int32_t n,
                         int32_t capacity, int32_t n_mb, int32_t policy, int32_t* out_assign,
                         int32_t* out_mb_tokens, int64_t* out_mb_cost_scaled,
                         int32_t* out_mb_max_len);

/* Heterogeneous parallel allocator, first step (Sec. 3.3): the pruned
 * parallelism configurations of one module. Encoders (backbone = 0) use data
 * and tensor parallelism, DP x TP devices; the backbone (backbone != 0) also
 * pipeline parallelism, DP x TP x PP devices. The section prunes
 * configurations whose DP does not divide the global batch, whose TP and PP
 * degrees fail to split the module's device budget, or whose tensor
 * parallelism spans two nodes; kept here:
 *  - DP divides global_batch;
 *  - DP*TP*PP <= devices (the module's device count, the product of its
 *    degrees, fits the cluster); for the backbone with layers > 0, PP also divides
 *    layers (pipeline stages of equal depth); layers = 0 drops that rule;
 *    PP = 1 for encoders;
 *  - TP divides per_node (TP groups on consecutive devices stay in one node).
 * Listed in increasing (DP, TP, PP) order into host int32
 * out_dp/out_tp/out_pp[cap] (any may be NULL); *out_n (host) receives the
 * count even when it exceeds cap (then EINVAL). Host only. Errors: EINVAL. */
fp_status alloc_candidates(int32_t backbone, int32_t devices, int32_t per_node, int32_t global_batch,
                           int32_t layers, int32_t* out_dp, int32_t* out_tp, int32_t* out_pp,
                           int32_t cap, int32_t* out_n);

/* Heterogeneous parallel allocator, flow matching (Eq. 1-2): pick one
 * configuration per module so that the devices used fit `budget` and
 * lexmax (G, -F), G = min(T_enc, T_bb), F = |T_enc - T_bb|, T_enc the sum of
 * the chosen encoder throughputs and T_bb the backbone's. Exact, on integer
 * throughputs (e.g. tokens/s from profiling); ties go to fewer devices, then
 * the smallest choice vector.
 *  n_modules   encoders followed by the backbone (>= 2)
 *  n_configs   host int32[n_modules], configurations per module (>= 1)
 *  tau, cost   host int64[sum(n_configs)], module by module: throughput and
 *              devices of each configuration
 * Outputs (host, may be NULL): out_choice int32[n_modules] configuration
 * index per module; out_G, out_F; out_devices (devices used).
 * Host only. Errors: EINVAL (also more than 2^22 encoder combinations),
 * ECAPACITY (no choice fits the budget). */
fp_status plan_allocation(int32_t n_modules, const int32_t* n_configs, const int64_t* tau,
                          const int64_t* cost, int64_t budget, int32_t* out_choice,
                          int64_t* out_G, int64_t* out_F, int64_t* out_devices);

/* Dynamic packing scheduler (Alg. 1, Sec. 3.4), host only (no pool, no GPU).
 * Phase 1, best fit: sequences are taken in input order; each goes to the open
 * microbatch whose residual capacity is the smallest that still holds it
 * (found by a segment tree over residuals [0, capacity]; equal residuals: the
 * microbatch opened first), else it opens a new microbatch of `capacity`
 * tokens; a microbatch whose residual falls below the shortest length of the
 * call is closed. Microbatches are numbered in the order they are opened.
 * Phase 2, load balancing: each microbatch's Eq. 3 cost, returned exactly as
 * capacity * sum(l) + l_max^2 (= capacity^2 * Cost); buckets of similar cost
 * by one-dimensional k-means (min(n_buckets, microbatches) centroids started
 * at the costs of sorted positions floor((2k+1) m / 2K), nearest centroid
 * with ties to the lower index, exact rational centroids, at most 100
 * rounds; bucket 0 holds the cheapest); buckets from the costliest down, each
 * one's microbatches in decreasing cost (ties: lower index) dealt to ranks
 * 0..N-1, then N-1..0, and so on, restarting at rank 0 for every bucket.
 *  lengths             host int32[n], each in [1, capacity]
 *  capacity            L, tokens per microbatch, at most 2^20
 *  n_ranks, n_buckets  N in [1, 2^20] data-parallel ranks, K >= 1 buckets
 * Outputs (host, caller-owned, any may be NULL; per-microbatch arrays need
 * room for n entries, of which *out_n_mb are written):
 *  out_mb_of_seq[n]    microbatch of each sequence
 *  out_mb_tokens, out_mb_max_len, out_mb_cost_scaled, out_mb_bucket,
 *  out_mb_rank         the rank a microbatch is dealt to
 *  out_mb_slot         its position in that rank's dispatch order
 * Deterministic. Errors: EINVAL. */
fp_status plan_dynamic_packing(const int32_t* lengths, int32_t n, int32_t capacity,
                               int32_t n_ranks, int32_t n_buckets, int32_t* out_mb_of_seq,
                               int32_t* out_n_mb, int32_t* out_mb_tokens, int32_t* out_mb_max_len,
                               int64_t* out_mb_cost_scaled, int32_t* out_mb_bucket,
                               int32_t* out_mb_rank, int32_t* out_mb_slot);

/* plan_dynamic_packing (Alg. 1, Sec. 3.4) over resident samples: sequence i is sample_ids[i]
 * with its pool length (text + image rows). Errors: EINVAL (also a sample
 * longer than capacity), ENOENT. */
fp_status plan_pool_packing(fp_pool* p, const uint64_t* sample_ids, int32_t n, int32_t capacity,
                            int32_t n_ranks, int32_t n_buckets, int32_t* out_mb_of_seq,
                            int32_t* out_n_mb, int32_t* out_mb_tokens, int32_t* out_mb_max_len,
                            int64_t* out_mb_cost_scaled, int32_t* out_mb_bucket,
                            int32_t* out_mb_rank, int32_t* out_mb_slot);

/* Consumer pack: the hot path (Sec. 3.1, Sec. 3.2). For samples
 * sample_ids[0..n) in order, writes the packed microbatch:
 *  out_emb           device bf16 [out_rows_cap, H], 16-byte aligned. Row
 *                    cu[k] + r holds row r of sample k: text rows are
 *                    embed_table[id] and image rows are the producer's rows,
 *                    interleaved as described at pool_write_sample. Rows
 *                    >= n_tokens are not touched.
 *  out_cu_seqlens    device int32[n+1] (or NULL): 0, l_0, l_0+l_1, ...
 *  out_position_ids  device int32[out_rows_cap] (or NULL): r within sample.
 *  embed_table       device bf16 [vocab, H], 16-byte aligned; may be NULL when
 *                    no sample has text. vocab must be >= the pool's vocab.
 *                    A table of at most 2.5 GiB is read with plain loads, which
 *                    let the device's memory-side cache keep its rows; a larger
 *                    one with non-temporal loads (this changes timing only).
 *  out_n_tokens, out_max_seqlen  host int32 (or NULL): total and longest l.
 *  tier_mask         FP_TIER_MASK_HBM copies text rows and rows on HBM pages
 *                    and writes cu_seqlens/position ids; FP_TIER_MASK_HOST
 *                    copies rows on host-tier pages; FP_TIER_MASK_ALL both.
 *                    Two launches with the two masks write what one ALL does.
 * Asynchronous on `stream`. Duplicated ids are packed twice. The row table
 * travels in the kernel arguments for up to 32 samples and 160 runs; a larger
 * microbatch's table is first copied to the device on `stream` from one of
 * the pool's pinned staging buffers.
 * Errors: EINVAL (also more than 1024 samples or images, or a microbatch of
 * more than 2^31 - 1024 16-byte vectors, i.e. n_tokens * 2H / 16), ENOENT,
 * ECAPACITY (sum of l > out_rows_cap), EALIGN, EHIP. */
fp_status pack_microbatch(fp_pool* p, const uint64_t* sample_ids, int32_t n,
                          const void* embed_table, int64_t vocab,
                          void* out_emb, int64_t out_rows_cap,
                          int32_t* out_cu_seqlens, int32_t* out_position_ids,
                          int32_t* out_n_tokens, int32_t* out_max_seqlen,
                          int32_t tier_mask, void* stream);

/* pack_microbatch for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same arguments, result and errors, but the call allocates nothing, host or
 * device, on success. A microbatch whose row table does not fit the kernel
 * arguments (more than 32 samples or 160 runs) has it copied, from one of the
 * staging buffers pool_create allocated, into a 64 KiB device scratch array
 * of the library, one per GPU, which holds the largest table a pack can have;
 * a larger table returns ECAPACITY (it cannot occur within the limits of
 * pack_microbatch). Every call on one GPU shares that array and leaves its
 * table there: calls that overlap on one GPU (on different streams, or
 * through different pools, with neither ordered after the other) race and
 * may read each other's table; calls in order on one stream do not. A sample
 * already packed on 8 other streams returns ESTATE when packed on a new one
 * (recording a 9th reader stream would grow a host list). */
fp_status pack_microbatch_noalloc(fp_pool* p, const uint64_t* sample_ids, int32_t n,
                                  const void* embed_table, int64_t vocab,
                                  void* out_emb, int64_t out_rows_cap,
                                  int32_t* out_cu_seqlens, int32_t* out_position_ids,
                                  int32_t* out_n_tokens, int32_t* out_max_seqlen,
                                  int32_t tier_mask, void* stream);

/* The library's (not an operation of the paper): lets the pool forget
 * `stream` before the caller destroys it: wherever the
 * pool remembers the stream as a reader of a sample (a pack ran there) or as
 * the stream of a sample's write, one event recorded now on the stream, after
 * the work queued there, takes its place (no event if the stream is idle).
 * Frees of those samples then wait for that event, not for the stream.
 * Not on a capturing stream. Errors: ESTATE, EHIP. */
fp_status pool_forget_stream(fp_pool* p, void* stream);

/* The library's (not an operation of the paper): ends the hold that
 * captured packs have on their samples (see HIP graphs
 * above): call it with a captured pack's sample id list (host uint64[n], in
 * any order; an id listed twice releases two captures of it) once no graph
 * holding that pack will be replayed again. Afterwards the samples may be
 * freed or migrated. All-or-nothing. Errors: ENOENT, EINVAL (an id holds
 * fewer captured packs than listed). */
fp_status pool_release_captured(fp_pool* p, const uint64_t* sample_ids, int32_t n);

/* Introspection (tests, benchmarks); host outputs, any may be NULL. */
fp_status pool_stats(const fp_pool* p, int64_t* free_hbm_pages, int64_t* free_host_pages,
                     int64_t* n_samples);

/* Page GVAs of a sample in visual-row order (Sec. 3.2: a sample's visual
 * embeddings are referenced by GVAs). gvas: host uint64[cap]; *n (host)
 * receives the page count even when cap is too small (then EINVAL). */
fp_status pool_sample_pages(const fp_pool* p, uint64_t sample_id, uint64_t* gvas,
                            int32_t cap, int32_t* n);

/* Sample metadata: *length = text + visual rows, *n_text, *n_vis (host, any NULL). */
fp_status pool_sample_info(const fp_pool* p, uint64_t sample_id, int32_t* length,
                           int32_t* n_text, int32_t* n_vis);

/* Translate a GVA through the page table (Sec. 3.2: translation is local to
 * the rank): *tier (FP_TIER_*) and *phys, the
 * device-visible address of that byte. Errors: EINVAL (unmapped GVA). */
fp_status pool_translate(const fp_pool* p, uint64_t gva, int32_t* tier, uint64_t* phys);

/* GVA layout (Sec. 3.2: per tier a region of world_size segments): region
 * starts and this rank's segment starts for the two tiers
 * (host uint64[2] each, may be NULL) and the page size in bytes. */
fp_status pool_layout(const fp_pool* p, uint64_t* region_start, uint64_t* segment_start,
                      int64_t* page_bytes);

/* Measurement aids (not steps of the method): plain kernels with the
 * pack's chunk geometry (chunks of 256 threads x 3 vectors of 16 bytes, or 2
 * for rows of 10 KiB or more, sized for the current device's compute units,
 * with the same shrinking tail chunks) and its load and store cache policy,
 * which move the bytes a pack moves and do nothing else, so a pack can be
 * timed against them in the same run. Asynchronous on `stream`, on the
 * calling thread's current device.
 *
 * fp_copy_bytes: copies `bytes` (a multiple of 16, at most (2^31 - 1024) * 16)
 * from device src to device dst, both 16-byte aligned, non-overlapping;
 * row_bytes (a multiple of 16) selects the chunk size a pack of such rows
 * uses. Errors: EINVAL, EALIGN, EHIP. */
fp_status fp_copy_bytes(const void* src, void* dst, int64_t bytes, int32_t row_bytes, void* stream);

/* fp_gather_rows: output row r (row_bytes bytes, a multiple of 16) of dst
 * (device, 16-byte aligned, n_rows * row_bytes bytes) is a copy of the
 * row_bytes bytes at address rows_src[r] with its low 4 bits cleared;
 * rows_src is a device uint64[n_rows] of device-readable, 16-byte aligned
 * addresses, which the call does not check (an invalid one faults the GPU).
 * Bit 0 of an entry marks an embedding-table row: a chunk of the output that
 * holds one reads with the loads pack_microbatch uses for table rows.
 * Errors: EINVAL, EALIGN, EHIP. */
fp_status fp_gather_rows(const uint64_t* rows_src, int32_t n_rows, int32_t row_bytes, void* dst, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FLOWPOOL_H */
