/* dv.h -- KV-cache streaming for one MI355X (gfx950): pack, unpack and swap.
 *
 * The operations are the data-movement core of the KV-cache streaming
 * library of "DejaVu: KV-cache Streaming for Fast, Fault-tolerant Generative
 * LLM Serving" (arXiv 2403.01876):
 *
 *   dv_stream_out_prompt  non-contiguous cache region -> one contiguous
 *                         buffer (the "scatter" primitive of Table 1, with
 *                         the buffered-copy optimisation of Sec. 4.1.1);
 *   dv_stream_out_token   the one-token increment of every layer after a
 *                         decode step (Sec. 4.1.1, Figure "cache_ft": each
 *                         step updates a small non-contiguous part);
 *   dv_stream_in          contiguous buffer -> a receiver's layout (the
 *                         "gather" primitive of Table 1; repopulating a lost
 *                         cache from its replica, Sec. 4.2.3);
 *   dv_swap_out/_in       microbatch swapping between a GPU slot and pinned
 *                         host memory (Sec. 4.2.2).
 *
 * Conventions shared by every call:
 *  - Return value: DV_OK (0) or a negative dv_status.  Arguments are checked
 *    on the host before anything is enqueued; on a validation error
 *    (DV_ERR_INVALID, _RANGE, _SPACE, _UNSUPPORTED) nothing is enqueued and no
 *    memory is touched.  DV_ERR_HIP means the runtime refused a launch or
 *    copy; a call that enqueues several (more than 64 sequences, split-key
 *    caches, ragged swaps, owner maps) may then have enqueued the ones
 *    before it, so the destination is unspecified until the call succeeds.
 *  - Asynchrony: work is enqueued on `stream` (a hipStream_t; NULL is the
 *    null stream) and is complete only once that stream has been
 *    synchronised.  Host arrays passed in (ranges, mb_base, block_table) are
 *    read during the call only and may be reused as soon as it returns.
 *  - Ownership: the caller owns every buffer (caches, contiguous buffers,
 *    block tables, host mirrors).  The library allocates nothing, keeps no
 *    state between calls and frees nothing.
 *  - Elements are opaque `elem_bytes`-byte words: results are bit copies
 *    (NaN payloads, -0 and subnormals preserved).
 *  - Aliasing: the source and destination of one call must not overlap
 *    (checked; DV_ERR_INVALID).
 *  - Thread safety: calls may be made from several host threads; calls on
 *    different streams that write the same bytes race, as any two kernels
 *    would.
 */
#ifndef DV_H
#define DV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* 2: dv_cache gained block_owner (the optional owner-map workspace).
 * 3: dv_stream_in_noalloc. */
#define DV_API_VERSION 3

/* The library is built with hidden visibility; only these calls export. */
#define DV_API __attribute__((visibility("default")))

typedef enum {
  DV_OK = 0,
  DV_ERR_INVALID = -1,     /* malformed descriptor or argument: null pointer, extent <= 0,
                              head_dim*elem_bytes not a multiple of 16, base not 16-byte
                              aligned, overlapping source and destination */
  DV_ERR_RANGE = -2,       /* microbatch/slot index, layer range or token range outside the
                              descriptor */
  DV_ERR_SPACE = -3,       /* destination capacity (or source size) below the stream size */
  DV_ERR_UNSUPPORTED = -4, /* well-formed but not handled: swap of a paged or split-key cache;
                              a split-key cache with more than 32 16-byte groups per token;
                              extents past the kernels' 32-bit index arithmetic -- more
                              than 2^24 layers, token
                              capacity (max_seq, or max_blocks*block_size) above 2^24,
                              head_dim*elem_bytes above 2^20 bytes, num_heads*head_dim*
                              elem_bytes above 2^24 bytes, capacity*head_dim*elem_bytes above
                              2^34 bytes, a paged block of one head (block_size*head_dim*
                              elem_bytes) above 2^33 bytes, a cache whose storage, or
                              whose stream of every layer and sequence at full capacity,
                              reaches 2^48 bytes,
                              or a launch whose grid would count 2^31 or more
                              tiles or 16-byte units (each launch covers up to 64
                              sequences; every launch of a call is checked first) */
  DV_ERR_HIP = -5          /* the HIP runtime refused to enqueue the work */
} dv_status;

typedef enum {
  DV_DENSE = 0,        /* [layer][K|V][batch][head][max_seq][head_dim] */
  DV_PAGED = 1,        /* pool [layer][K|V][num_blocks][head][block_size][head_dim], tokens
                          reach blocks through a per-sequence block table */
  DV_DENSE_KSPLIT = 2  /* as DV_DENSE, except the key half stores head_dim in 16-byte groups
                          outside the token axis: [layer][K][batch][head][head_dim/x][max_seq][x],
                          x = 16/elem_bytes (the split-key layout of decoder kernels that
                          read keys 16 bytes at a time); the value half is dense */
} dv_kind;

typedef enum { DV_MEM_DEVICE = 0, DV_MEM_HOST_PINNED = 1 } dv_mem;

/* A KV-cache layout and where its microbatches live.  A cache holds one
 * pipeline stage's layers and one tensor-parallel shard's heads, so
 * num_layers and num_heads are local counts.  Logical element
 * X(l, kv, b, h, s, d) -- layer l, kv 0 = key / 1 = value, sequence b, head
 * h, token s, dimension d -- is stored at element index
 *   DV_DENSE  ((((l*2+kv)*batch + b)*num_heads + h)*max_seq + s)*head_dim + d
 *   DV_PAGED  ((((l*2+kv)*num_blocks + T[b][s/block_size])*num_heads + h)*block_size
 *              + s%block_size)*head_dim + d,      T = block_table[mb]
 *   DV_DENSE_KSPLIT, kv = 0:
 *             (((((l*2)*batch + b)*num_heads + h)*(head_dim/x) + d/x)*max_seq + s)*x + d%x
 * of microbatch mb's base address mb_base[mb].  All bases 16-byte aligned. */
typedef struct dv_cache {
  int32_t kind;        /* dv_kind */
  int32_t mem;         /* dv_mem: where the cache bytes live (swap direction checks) */
  int32_t elem_bytes;  /* bytes per element (2 for fp16/bf16) */
  int32_t num_layers;  /* layers held */
  int32_t num_heads;   /* KV heads held */
  int32_t head_dim;    /* head_dim * elem_bytes must be a multiple of 16 */
  int32_t batch;       /* sequences per microbatch */
  int32_t max_seq;     /* dense kinds: token capacity per sequence; paged: ignored
                          (capacity is max_blocks * block_size) */
  int32_t block_size;  /* paged: tokens per block */
  int32_t num_blocks;  /* paged: blocks in each microbatch's pool */
  int32_t max_blocks;  /* paged: columns of each block table */
  int32_t num_mb;      /* entries of mb_base (and block_table) */
  void* const* mb_base;              /* host array [num_mb] of cache base addresses */
  const int32_t* const* block_table; /* paged: host array [num_mb] of device addresses of
                                        int32 [batch][max_blocks] tables; an entry outside
                                        [0, num_blocks) marks an unmapped block.  A table
                                        must not overlap anything a call writes (stream
                                        destination, pool on stream-in, owner map, claim
                                        counts): DV_ERR_INVALID */
  int32_t* const* block_owner;       /* paged, optional (NULL, or NULL entries, to leave
                                        unused): host array [num_mb] of device addresses of
                                        caller-owned int32 [num_blocks] workspaces, 4-byte
                                        aligned; see dv_stream_in */
} dv_cache;

/* The contiguous buffer ("wire") a stream produces or consumes, for layer
 * range [l0, l1) and per-sequence token ranges [t0[b], t1[b]):
 *   n_b = t1[b] - t0[b],  P_b = sum_{b' < b} n_b',  N = sum_b n_b,
 *   X(l,kv,b,h,s,d) sits at element
 *   ((l-l0)*2 + kv)*N*H*D + P_b*H*D + h*n_b*D + (s - t0[b])*D + d,
 * i.e. [layer][K|V][sequence][head][token][head_dim] with ragged sequences,
 * (l1-l0)*2*H*D*N*elem_bytes bytes in all.  It is headerless: the receiver
 * passes the same ranges.  Layer ranges concatenate: the buffer of [l0, l1)
 * is that of [l0, m) followed by that of [m, l1), so a prompt can be
 * streamed layer by layer as each layer is computed (Sec. 4.1.1,
 * optimisation 2). */

/* Storage bytes of one microbatch of `c` (dense: L*2*B*H*S*D*E; paged:
 * L*2*NB*H*bs*D*E).  Host-only.  DV_OK, DV_ERR_INVALID, DV_ERR_UNSUPPORTED
 * (extents past the limits listed with DV_ERR_UNSUPPORTED). */
DV_API int dv_cache_bytes(const dv_cache* c, uint64_t* out_bytes);

/* Bytes of the contiguous buffer for these ranges (formula above).  t0 may
 * be NULL (all zero).  Host-only.  DV_OK, DV_ERR_INVALID, DV_ERR_RANGE,
 * DV_ERR_UNSUPPORTED. */
DV_API int dv_packed_bytes(const dv_cache* c, int32_t l0, int32_t l1, const int32_t* t0,
                    const int32_t* t1, uint64_t* out_bytes);

/* Pack microbatch `mb` of `src`, layers [l0, l1), tokens [t0[b], t1[b]) of
 * each sequence b, into `dst` in the wire order above.  A prompt stream
 * passes t0 = NULL (or zeros) and t1 = prompt lengths; a whole-cache replica
 * passes the valid lengths; an empty range (t0[b] == t1[b]) skips a
 * sequence (e.g. a request that stopped early).  `dst` is device memory (or
 * any memory kernels may write) of `dst_cap` bytes, 16-byte aligned.  On
 * return *out_bytes (if not NULL) holds the stream size, also on
 * DV_ERR_SPACE.  Paged caches: tokens whose table entry is outside
 * [0, num_blocks) are rejected by no host check (the table is on the
 * device); the kernel skips them and their wire bytes are left unwritten.
 * DV_OK, DV_ERR_INVALID, DV_ERR_RANGE, DV_ERR_SPACE, DV_ERR_UNSUPPORTED,
 * DV_ERR_HIP. */
DV_API int dv_stream_out_prompt(const dv_cache* src, int32_t mb, int32_t l0, int32_t l1,
                         const int32_t* t0, const int32_t* t1, void* dst, uint64_t dst_cap,
                         uint64_t* out_bytes, void* stream);

/* Pack the decode-step increment: token pos[b] of every sequence, layers
 * [l0, l1); pos[b] < 0 marks an inactive sequence (contributes nothing).
 * Identical to dv_stream_out_prompt with t0 = pos, t1 = pos + 1 (0 tokens
 * for inactive sequences), so the wire is [layer][K|V][active seq][head][D].
 * Same arguments, errors and ownership as dv_stream_out_prompt. */
DV_API int dv_stream_out_token(const dv_cache* src, int32_t mb, int32_t l0, int32_t l1,
                        const int32_t* pos, void* dst, uint64_t dst_cap, uint64_t* out_bytes,
                        void* stream);

/* Unpack `src` (a wire of exactly dv_packed_bytes bytes for these ranges;
 * `src_bytes` must be at least that) into microbatch `mb` of `dst`.  Only the
 * streamed positions are written; every other byte of the cache is left as
 * it was.  The receiver layout may differ from the sender's (capacity,
 * dense vs paged vs split-key).  Paged receivers: tables must map distinct
 * tokens to distinct slots (the same block must not appear twice within the
 * streamed ranges), else the result is whichever write lands last; tokens
 * with an unmapped entry are skipped.  A token increment is streamed in with
 * t0 = pos, t1 = pos + 1.
 *
 * Paged receivers with a block_owner workspace for `mb`: when some
 * sequence's run per head is longer than 4 KB (shorter runs go through a
 * kernel that moves one 16-byte unit per lane in stream order), the call
 * has at most 256 sequences and fewer than 2^31 tokens, and it writes at
 * least five ninths of the pool's blocks, the library first rebuilds in the
 * workspace the inverse of the table over the streamed ranges (pool block
 * -> sequence * max_blocks + logical block, -1 for blocks not written) and
 * then writes the pool in physical block order in one launch, so the
 * writes are sequential instead of scattered
 * by the table (measured on MI355X: 69 % -> 75 % of HBM peak for the
 * LLaMA-2-70B stage's pool; below about five ninths of the blocks, the
 * workgroups that find no block to write cost more than that gains).  The bytes
 * written are the same either way.  The workspace must not overlap the
 * cache or `src` (DV_ERR_INVALID); its contents are scratch between calls,
 * and calls that scatter into the same microbatch must not overlap in time.
 * DV_OK, DV_ERR_INVALID, DV_ERR_RANGE, DV_ERR_SPACE, DV_ERR_UNSUPPORTED,
 * DV_ERR_HIP. */
DV_API int dv_stream_in(const dv_cache* dst, int32_t mb, int32_t l0, int32_t l1, const int32_t* t0,
                 const int32_t* t1, const void* src, uint64_t src_bytes, void* stream);

/* dv_stream_in for callers that cannot allocate and so can pass no owner-map
 * workspace: code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation.  Identical to dv_stream_in (same arguments,
 * results, conditions for the pool-order scatter and errors), except that a
 * paged receiver's owner map is built in a buffer of the library's own
 * instead of dst->block_owner, which is ignored: a static device array of
 * DV_NOALLOC_MAX_BLOCKS int32 entries (4 MiB), one per GPU, reserved when
 * the library's code object is first loaded on that GPU and held until the
 * process ends.  The call allocates nothing (no hipMalloc, no allocating
 * library routine); its first call on a device looks the array's address up
 * there once.  The current device's array is used, so `stream` must belong
 * to the current device; a paged receiver's call on a stream of another
 * device is refused with DV_ERR_INVALID before anything is enqueued.  Paged
 * receivers with more than
 * DV_NOALLOC_MAX_BLOCKS blocks are refused with DV_ERR_UNSUPPORTED before
 * anything is enqueued.  Every call that uses the array rebuilds the map in
 * it (cleared by a kernel, then filled), so nothing carries over from the
 * previous call; but all calls on one GPU share that GPU's array, so two
 * calls whose work overlaps in time on one GPU (different streams, or
 * different host threads) race on it and leave their pools undefined --
 * order them on one stream or synchronise between them.  Dense and
 * split-key receivers use no buffer and behave exactly as dv_stream_in.
 * DV_OK, DV_ERR_INVALID, DV_ERR_RANGE, DV_ERR_SPACE, DV_ERR_UNSUPPORTED,
 * DV_ERR_HIP. */
#define DV_NOALLOC_MAX_BLOCKS (1 << 20)
DV_API int dv_stream_in_noalloc(const dv_cache* dst, int32_t mb, int32_t l0, int32_t l1,
                                const int32_t* t0, const int32_t* t1, const void* src,
                                uint64_t src_bytes, void* stream);

/* Debug check of a paged table over token ranges [t0[b], t1[b]) (t0 may be
 * NULL): writes to `counts` (device int32 [num_blocks], caller owned,
 * 4-byte aligned, disjoint from the pool) how many (sequence, logical
 * block) entries that hold a streamed token map to each pool block.  A
 * count above 1 marks a block that dv_stream_in would write twice, which
 * the paged receivers' precondition rules out; entries outside
 * [0, num_blocks) are not counted.  Enqueued on `stream` (two small
 * launches); read `counts` after synchronising it.
 * DV_OK, DV_ERR_INVALID, DV_ERR_RANGE, DV_ERR_UNSUPPORTED (not DV_PAGED),
 * DV_ERR_HIP. */
DV_API int dv_block_claims(const dv_cache* c, int32_t mb, const int32_t* t0, const int32_t* t1,
                           int32_t* counts, void* stream);

/* Microbatch swap-out: copy layers [l0, l1), tokens [t0[b], t1[b]) of device
 * slot `slot` of `dev` to host microbatch `host_mb` of `host`, at equal
 * logical coordinates; all other host bytes are left as they were.  Both
 * caches must be DV_DENSE with equal num_layers, num_heads, head_dim, batch
 * and elem_bytes (their max_seq may differ); `dev` must be DV_MEM_DEVICE and
 * `host` DV_MEM_HOST_PINNED (allocated with hipHostMalloc, which kernels can
 * address).  Rows of 64 KB or more (one sequence's tokens of one head) move
 * on the DMA engines (hipMemcpy2DAsync over the token rows) on `stream`, so
 * they overlap kernels on other streams; narrower rows -- a decode step's
 * update is one 256-byte row per (layer, K|V, sequence, head) -- are copied
 * by one kernel on `stream` that writes the pinned mirror directly.
 * Swapping a whole microbatch passes its valid lengths; the step-t update
 * passes t0 = t, t1 = t + 1.
 * DV_OK, DV_ERR_INVALID, DV_ERR_RANGE, DV_ERR_UNSUPPORTED, DV_ERR_HIP. */
DV_API int dv_swap_out(const dv_cache* dev, int32_t slot, const dv_cache* host, int32_t host_mb,
                int32_t l0, int32_t l1, const int32_t* t0, const int32_t* t1, void* stream);

/* Microbatch swap-in (prefetch): the reverse copy, host microbatch
 * `host_mb` -> device slot `slot`.  Same rules as dv_swap_out. */
DV_API int dv_swap_in(const dv_cache* host, int32_t host_mb, const dv_cache* dev, int32_t slot,
               int32_t l0, int32_t l1, const int32_t* t0, const int32_t* t1, void* stream);

/* ------------------------------------------------------------------------
 * Microbatch swap scheduler (Sec. 4.2.2, Figure "swapping").  The caches of
 * all D microbatches live in pinned host memory (`host`, num_mb = D); two
 * device slots (`dev_slots`, the first two mb_base entries) hold the
 * microbatch being processed and the next one.  Per step of microbatch x:
 *   dv_swapper_prefetch(x+1, len)      swap-in of x+1 into the other slot on
 *                                      the scheduler's input stream, once that
 *                                      slot's previous occupant has been
 *                                      swapped out;
 *   dv_swapper_begin_step(x, stream)   makes `stream` wait until x is in its
 *                                      slot; returns the slot for the step;
 *   ... the step writes the slot on `stream` ...
 *   dv_swapper_end_step(x, stream, t0, t1)
 *                                      after the work queued on `stream`, swap
 *                                      out the part the step updated (tokens
 *                                      [t0[b], t1[b]), e.g. the one new token)
 *                                      on the scheduler's output stream.
 * Slots are dealt alternately in prefetch order.  The calls keep the slot
 * bookkeeping and hand each swap to a worker thread, which waits on the host
 * for what the swap depends on (the step, before a swap-out; the slot's
 * previous swap-out, before a swap-in) and then issues it, so that only the
 * compute stream waits on the GPU, for residency (streams waiting on the GPU
 * behind a swap-in stretched it by about 0.46 ms each on MI355X).
 * begin_step blocks the host until the worker has issued that microbatch's
 * swap-in; end_step blocks only if 8 swap-outs are still waiting for their
 * steps.  create allocates four streams, twelve events and the worker thread
 * (the only allocations);
 * the descriptors' base arrays are copied.  Overlap needs the scheduler's
 * streams on hardware queues other than the compute stream's: HIP deals
 * ordinary streams onto a pool of GPU_MAX_HW_QUEUES hardware queues (4 by
 * default) and streams sharing a queue execute in order.  The input and the
 * output stream therefore each come in two forms: one with a hardware queue
 * of its own (a CU-masked stream over every CU, which HIP never shares), used
 * when the compute stream of the latest begin_step / end_step is not the
 * legacy null stream, and one from the shared pool, used otherwise (HIP
 * makes CU-masked streams wait for the null stream).  With the null stream
 * as compute stream a process with many streams should raise
 * GPU_MAX_HW_QUEUES, or compute on a stream of its own (measured on MI355X:
 * a pooled stream landed on the compute stream's queue in one creation of
 * four; the own-queue form never did).  Both
 * caches DV_DENSE with equal shapes (capacities may differ), dev in
 * DV_MEM_DEVICE, host in DV_MEM_HOST_PINNED; the two slots must be disjoint
 * and so must the host mirrors (create returns DV_ERR_INVALID otherwise).
 * One scheduler per host thread.
 * prefetch and end_step check their ranges against both the slots and the
 * host mirrors before enqueuing anything; a refused call changes nothing.
 * begin_step and end_step refuse a compute stream under graph capture
 * (DV_ERR_INVALID): the scheduler's streams wait on events the caller's
 * stream records, which a capture would only turn into graph nodes.
 * Errors: DV_ERR_INVALID (bad arguments; prefetch into a slot whose
 * occupant's step has not ended), DV_ERR_RANGE (microbatch outside `host`;
 * begin/end of a microbatch not prefetched; ranges that do not fit),
 * DV_ERR_UNSUPPORTED, DV_ERR_HIP. */
typedef struct dv_swapper dv_swapper;
DV_API int dv_swapper_create(const dv_cache* dev_slots, const dv_cache* host, dv_swapper** out);
DV_API int dv_swapper_prefetch(dv_swapper* s, int32_t mb, const int32_t* len);
DV_API int dv_swapper_begin_step(dv_swapper* s, int32_t mb, void* compute_stream, int32_t* slot_out);
DV_API int dv_swapper_end_step(dv_swapper* s, int32_t mb, void* compute_stream, const int32_t* t0,
                        const int32_t* t1);
/* Waits for all swaps queued so far. */
DV_API int dv_swapper_sync(dv_swapper* s);
/* Waits for queued swaps, then frees the scheduler's streams and events. */
DV_API int dv_swapper_destroy(dv_swapper* s);

/* ------------------------------------------------------------------------
 * Background streamer: layer-by-layer prompt streaming and token streaming
 * in parallel with computation, driven by a background host thread
 * (Sec. 4.1.1, optimisations 2 and 3).  The compute thread calls
 * dv_streamer_push after queuing the work that produces a region on its
 * compute stream; push records an event there and returns.  A worker thread
 * waits for that event on the host (no cross-stream wait is queued on the
 * GPU) and then, on the streamer's own stream: packs the region
 * (layers [l0, l1), tokens [t0[b], t1[b]) of microbatch `mb` of `src`, t0 may
 * be NULL) into `staging` + staging_offset with dv_stream_out_prompt, and
 * copies the packed bytes to `dst` + dst_offset (pinned host memory, or
 * device memory; a host destination is written by pitched copies, which run
 * on the SDMA engines and leave the compute units to the compute stream,
 * where a plain copy would run as a blit kernel on them).  From a DV_DENSE
 * source whose longest (sequence, head) run in the region is 64 KB or more,
 * a host destination is filled by the SDMA engines straight from the cache
 * (pitched copies over the heads' runs, no kernel and no staging).  Offsets are the
 * caller's: pushing a prompt's layers one by one at offsets that accumulate
 * their sizes leaves the whole prompt's contiguous buffer in `dst`, since
 * layer ranges concatenate; decode steps can cycle through a few staging
 * slots while filling a long host log.
 * Pushes run in push order.  `staging` (device) and `dst` are caller owned,
 * disjoint from each other, from the source microbatch and from a paged
 * source's block table (create returns DV_ERR_INVALID otherwise); offsets
 * 16-byte aligned, each must hold its offset + bytes (else DV_ERR_SPACE).
 * create allocates two side streams (one with a hardware queue of its own,
 * used for pushes from any compute stream but the legacy null stream, and
 * one from HIP's shared pool for pushes from the null stream; see the swap
 * scheduler), 64 events and the worker thread; push blocks only when 64
 * pushes are waiting for the worker.  flush blocks until everything pushed
 * has reached `dst` and returns the first error the worker met (a later
 * push also returns it).  destroy drains, then frees.  Same alignment,
 * range and layout rules as dv_stream_out_prompt.  push refuses a compute
 * stream under graph capture (DV_ERR_INVALID, nothing recorded): the worker
 * waits on the host for the event push records, which a capture would only
 * turn into a graph node. */
typedef struct dv_streamer dv_streamer;
DV_API int dv_streamer_create(const dv_cache* src, int32_t mb, void* staging, uint64_t staging_cap,
                       void* dst, uint64_t dst_cap, dv_streamer** out);
DV_API int dv_streamer_push(dv_streamer* s, void* compute_stream, int32_t l0, int32_t l1,
                            const int32_t* t0, const int32_t* t1, uint64_t staging_offset,
                            uint64_t dst_offset, uint64_t* out_bytes);
DV_API int dv_streamer_flush(dv_streamer* s);
DV_API int dv_streamer_destroy(dv_streamer* s);

/* Static text for a dv_status value. */
DV_API const char* dv_status_string(int status);

/* DV_API_VERSION of the built library. */
DV_API int dv_api_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DV_H */
