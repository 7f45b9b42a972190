/*
 * agnes.h -- C ABI of the MI355X (gfx950) hyperbatch GNN data-preparation library.
 *
 * Implements the data-preparation path of AGNES (arXiv 2601.01473): multi-hop
 * neighbour sampling and feature-row gathering for H minibatches at once, with
 * the requests of every minibatch bucketed by fixed-size storage block so that
 * each block serves all the requests that fall in it (Sec. 3.3, Sec. 3.4(3),
 * Alg. 1).  Blocks are pages resident in HBM.
 *
 * Conventions shared by every entry point:
 *   - Return value: AGNES_OK or an error code; on error every out-handle is set
 *     to NULL and agnes_last_error() describes the failure.  No exception, abort
 *     or exit crosses this boundary.
 *   - "host" pointers are ordinary CPU memory; "device" pointers are HIP device
 *     memory of the current device.
 *   - hip_stream is a hipStream_t passed as void* (NULL = the null stream).
 *   - All node ids are int32 in [0, num_nodes); num_nodes < 2^31.
 *
 * Environment variables read by the library (none changes any result):
 *   - AGNES_DEBUG_SYNC=1: every kernel launch synchronises its stream and
 *     checks for an error right after it (outside graph capture), so a fault
 *     is reported at the launch that caused it.  Read once per process.
 *   - AGNES_WIDE_OFFSETS=1: agnes_build_blocks* keep int64 CSR offsets 64-bit
 *     on the device; by default the offsets of a graph with fewer than 2^31
 *     edges are stored as int32.  Read at every build.
 */
#ifndef AGNES_H
#define AGNES_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    AGNES_OK = 0,
    AGNES_ERR_INVALID = 1,   /* bad argument or input content */
    AGNES_ERR_NOMEM = 2,     /* device or host allocation failed */
    AGNES_ERR_DEVICE = 3,    /* a HIP call failed; the HIP error string is in last-error */
    AGNES_ERR_RANGE = 4,     /* a per-minibatch count or a total exceeds 2^31 - 1 */
    AGNES_ERR_INTERNAL = 5
} agnes_status;

typedef enum {
    AGNES_INT32 = 0,
    AGNES_INT64 = 1,
    AGNES_FLOAT32 = 2,
    AGNES_FLOAT16 = 3,
    AGNES_BFLOAT16 = 4
} agnes_dtype;

typedef struct agnes_store agnes_store;   /* opaque: HBM-resident topology/feature blocks */
typedef struct agnes_batch agnes_batch;   /* opaque: device outputs of one hyperbatch */

/* Graph topology in CSR form with source rows (host memory, read only).
 * offsets: num_nodes+1 entries of offsets_dtype (AGNES_INT32 or AGNES_INT64),
 *          offsets[0] = 0, nondecreasing, offsets[num_nodes] = num_edges.
 * indices: num_edges int32 neighbour ids, each in [0, num_nodes).  A row's order
 *          is the order in which its neighbours are numbered (positions). */
typedef struct {
    int64_t num_nodes;
    int64_t num_edges;
    agnes_dtype offsets_dtype;
    const void* offsets;
    const int32_t* indices;
} agnes_csr;

/* Node features (host memory, read only): num_nodes rows of dim elements,
 * row-major.  The rows are moved as opaque bytes: row_bytes = dim * size(dtype),
 * which must be a multiple of 4. */
typedef struct {
    const void* data;
    int64_t dim;
    agnes_dtype dtype;   /* AGNES_FLOAT32, AGNES_FLOAT16 or AGNES_BFLOAT16 */
} agnes_features;

/*
 * Build the block store (Sec. 3.2(1) storage layer; Sec. 3.2(2) object index
 * table).  The CSR index array is cut into topology blocks of block_bytes/4
 * edges; a node's object is its adjacency list and its home block is the block
 * holding its first edge, so objects sit in ascending node order and a long list
 * continues into the following blocks.  The feature matrix is cut into feature
 * blocks of floor(block_bytes / row_bytes) rows.  The object index table keeps,
 * per topology block, the first and last node whose home it is.
 *
 * csr, feat: host inputs, copied into library-owned HBM; the caller may free
 *            them once the call returns.
 * block_bytes: power of two in [16, 2^24] and >= row_bytes.
 * hip_stream: stream used for the uploads; the call returns after they finish.
 * out: receives the store; release it with agnes_free().
 * Errors: INVALID (null pointer, non-monotone offsets, offsets[N] != E, index
 * out of range, num_nodes >= 2^31, bad dtype, row_bytes % 4 != 0, bad
 * block_bytes), NOMEM, DEVICE.
 */
agnes_status agnes_build_blocks(const agnes_csr* csr, const agnes_features* feat,
                                uint64_t block_bytes, void* hip_stream, agnes_store** out);

/*
 * Prepare one hyperbatch (Alg. 1): for each of the H minibatches (row j of
 * targets, global minibatch index m = mb_base + j) run L hops of neighbour
 * sampling, then gather the feature rows of every sampled node.
 *
 * Hop l (fanout f_l = fanouts[l], l = 0 nearest the targets): every node already
 * in minibatch j is a request; it receives min(deg, f_l) distinct neighbours,
 * drawn uniformly without replacement by Floyd's algorithm from Philox4x64-10
 * words at key (seed, 0), counter (i >> 2, v, m, l), word i taking lane i & 3,
 * integer draws floor(w * n / 2^64), listed in ascending edge position.  The
 * minibatch's node list grows by the sampled neighbours not yet in it, in
 * ascending global id (targets first, in the given order).  Hop l is emitted as
 * a CSR block: one row per node present before the hop, columns in local ids.
 * Requests are served block by block: the frontier of all minibatches is
 * bucketed by topology block (the bucket matrix Bck of Sec. 3.4(3)) and each
 * block's requests are sampled together; the gather is bucketed by feature
 * block the same way (Alg. 1, gathering loop).  Results depend only on
 * (store, targets, fanouts, seed, mb_base), not on the bucketing, the launch
 * geometry or how minibatches are grouped into hyperbatches.
 *
 * targets: HOST int32 [H][B] (Alg. 1's input N, row j = minibatch j); distinct
 * within each row, each in [0, N).  The call copies them (through a pinned
 * staging buffer owned by the batch) to the device on hip_stream, so the
 * caller may reuse the array as soon as the call returns.
 * H in [1, 4096], B >= 1, L in [1, AGNES_MAX_LAYERS], fanouts: host int32 [L],
 * each in [0, 1024].  seed: any 64-bit value.  mb_base >= 0.
 * Every hop's requests plus sampled edges must stay below 2^32 in the worst
 * case: H * cap_l * (1 + f_l) < 2^32, where cap_0 = B and cap_{l+1} =
 * min(cap_l * (1 + f_l), max(num_nodes, B)); otherwise AGNES_ERR_RANGE is
 * returned before anything is allocated or enqueued.
 * out: if *out is NULL a new batch is created; if it holds a batch previously
 *      returned for the same store, that batch's device buffers are reused (and
 *      grown when needed) and its previous contents are overwritten.
 * The call enqueues on hip_stream and returns when the outputs are complete.
 * Each batch owns the scratch memory of its hyperbatch, so several batches can
 * be in flight on one store.
 * Errors: INVALID (bad sizes, target out of range or duplicated within a
 * minibatch), RANGE (a minibatch with >= 2^31 nodes or edges, or the 2^32
 * bound above), NOMEM, DEVICE.
 * On error *out is NULL and a batch passed in is released.
 */
agnes_status agnes_hyperbatch_prepare(agnes_store* store, const int32_t* targets, int32_t H,
                                      int32_t B, const int32_t* fanouts, int32_t L,
                                      uint64_t seed, int64_t mb_base, void* hip_stream,
                                      agnes_batch** out);

/* The same with the targets already in DEVICE memory (int32 [H][B] on the
 * store's device; read by kernels on hip_stream, so they must stay valid until
 * the call returns).  No host copy or upload is made. */
agnes_status agnes_hyperbatch_prepare_device(agnes_store* store, const int32_t* targets, int32_t H,
                                             int32_t B, const int32_t* fanouts, int32_t L,
                                             uint64_t seed, int64_t mb_base, void* hip_stream,
                                             agnes_batch** out);

/*
 * The same hyperbatch in two steps, so that the sampling of one hyperbatch can
 * run while the gather of another streams rows (Sec. 3.4(4): work continues
 * while data moves).  agnes_hyperbatch_prepare = begin + finish + wait.
 *
 * agnes_hyperbatch_begin: same arguments and checks as prepare (HOST targets,
 *   copied by the call); enqueues their upload and the L sampling hops on
 *   hip_stream and returns without waiting.  A batch that is still
 *   gathering from an earlier hyperbatch may be passed in: the call first waits
 *   for that gather; the batch's previous views become invalid.
 * agnes_batch_finish: waits on the host for the output sizes of the begun
 *   hyperbatch, sizes the outputs, and enqueues the gather on hip_stream (which
 *   may differ from the begin stream; it is ordered after the sampling).  Returns
 *   without waiting for the gather.  Views are valid after this call; device
 *   contents after agnes_batch_wait (or once hip_stream has been synchronised).
 *   Errors (INVALID targets, RANGE) leave the batch empty and reusable.
 * agnes_batch_wait: blocks until the batch's outputs and statistics are complete.
 */
agnes_status agnes_hyperbatch_begin(agnes_store* store, const int32_t* targets, int32_t H,
                                    int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed,
                                    int64_t mb_base, void* hip_stream, agnes_batch** out);
/* agnes_hyperbatch_begin_device: the same with DEVICE targets, which must stay
 *   valid until the hyperbatch is finished. */
agnes_status agnes_hyperbatch_begin_device(agnes_store* store, const int32_t* targets, int32_t H,
                                           int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed,
                                           int64_t mb_base, void* hip_stream, agnes_batch** out);
agnes_status agnes_batch_finish(agnes_batch* batch, void* hip_stream);
agnes_status agnes_batch_wait(agnes_batch* batch);

#define AGNES_MAX_LAYERS 8

/* Read-only view of a batch: Alg. 1's outputs, the sampled node set N_s of
 * every minibatch (nodes, with the per-hop CSR blocks that the sampling loop
 * builds) and the gathered feature rows F_g (features, the gathering loop's
 * output), together with the offsets that locate each minibatch in them.
 * Host arrays stay valid until the batch is freed or reused; device arrays
 * likewise.  Fails with AGNES_ERR_INVALID for a batch whose hyperbatch has not
 * been finished (agnes_batch_finish or prepare); ownership stays with the batch.
 *   node_off[H+1]: minibatch j owns nodes[node_off[j] .. node_off[j+1]) and the
 *                  same rows of features.
 *   layer_sizes[H*(L+1)]: |D_0| = B, then the node count after each hop.
 *   nodes (device int32): global ids in local-id order, minibatch-major.
 *   rp_off[l][H+1], row_ptr[l] (device int32): hop l's row pointers of minibatch
 *                  j are row_ptr[l][rp_off[l][j] .. +layer_sizes[j][l]+1), from 0.
 *   col_off[l][H+1], col[l] (device int32): hop l's columns of minibatch j are
 *                  col[l][col_off[l][j] .. col_off[l][j+1]), local ids.
 *   features (device): [node_off[H]][row_bytes] gathered rows. */
typedef struct {
    int32_t H, L;
    int64_t row_bytes;
    const int64_t* node_off;
    const int32_t* layer_sizes;
    const int32_t* nodes;
    const int64_t* rp_off[AGNES_MAX_LAYERS];
    const int32_t* row_ptr[AGNES_MAX_LAYERS];
    const int64_t* col_off[AGNES_MAX_LAYERS];
    const int32_t* col[AGNES_MAX_LAYERS];
    const void* features;
} agnes_batch_view;

agnes_status agnes_batch_view_get(const agnes_batch* batch, agnes_batch_view* out);

/* Exact integer statistics of a prepared hyperbatch and the device time of
 * each phase when profiling is on (else -1).  Per hop l: requests R_l (the
 * nodes of every minibatch that the hop samples from), sampled edges S_l, new
 * nodes U_l, and T_l, the non-empty rows of the bucket matrix Bck (Sec. 3.4(3):
 * one row per topology block, the topology blocks the hop loads in Alg. 1's
 * sampling loop); then the gathered rows sum_j |N_j|, the distinct rows among
 * them, and the non-empty feature-block rows (the feature blocks Alg. 1's
 * gathering loop loads).  Waits for the batch; out is caller-owned.  Fails
 * with AGNES_ERR_INVALID for a batch with no finished hyperbatch. */
typedef struct {
    int32_t L;
    int64_t requests[AGNES_MAX_LAYERS];
    int64_t sampled[AGNES_MAX_LAYERS];
    int64_t new_nodes[AGNES_MAX_LAYERS];
    int64_t topo_blocks[AGNES_MAX_LAYERS];
    int64_t rows;
    int64_t distinct_rows;
    int64_t feat_blocks;
    float sample_ms;     /* all hops: bucketing, sampling, dedupe, relabel */
    float gather_ms;     /* gather bucketing and row copy */
    float copy_ms;       /* the row-copy kernel alone */
} agnes_stats;

agnes_status agnes_batch_stats(const agnes_batch* batch, agnes_stats* out);   /* waits for the batch */

/* The sampler's random-number generator, Philox4x64-10 (Sec. 3.4(3): every
 * request's draws come from a counter-based generator keyed by the request),
 * evaluated by the device code the sampler uses, for checking it against the
 * generator's published definition.  counters: host [n][4], keys: host [n][2],
 * out: host [n][4] (the four output words of each pair); n >= 0.  Runs on the
 * current device and waits for the result.  The sampler's draw i of request
 * (node v, minibatch m, hop l) is word i % 4 of counter (i / 4, v, m, l) and
 * key (seed, 0). */
agnes_status agnes_philox4x64_10(const uint64_t* counters, const uint64_t* keys, int64_t n, uint64_t* out);

/* Device memory allocator.  By default the library allocates its device
 * memory (stores, batches, their scratch space and outputs) with hipMalloc and
 * frees it with hipFree.  A caller that wants its own allocator to own that
 * memory (e.g. a framework's caching allocator) installs two callbacks:
 *   alloc(bytes, user) returns device memory of the current device, aligned
 *     to 256 bytes, or NULL on failure (the library call then fails with
 *     AGNES_ERR_NOMEM; a misaligned block is released and AGNES_ERR_INVALID
 *     returned);
 *   release(ptr, bytes, user) takes back a block that alloc returned.  The
 *     library calls it only after every piece of work it enqueued on that
 *     block's device has completed (it synchronises the device first, as
 *     hipFree does), so the block may be reused at once.
 * Both callbacks non-NULL installs them, both NULL restores hipMalloc / hipFree,
 * anything else is AGNES_ERR_INVALID.  The setting is process-wide and applies
 * to allocations made after the call; each block is released through the
 * callback that pairs with the allocator it came from, whatever is installed
 * by then.  Install it before the library's other calls, not concurrently with
 * them.  Allocations happen when a store is built and when a batch's buffers
 * grow (the first hyperbatches of a shape); pinned host memory is not affected. */
typedef void* (*agnes_device_alloc_fn)(uint64_t bytes, void* user);
typedef void (*agnes_device_free_fn)(void* ptr, uint64_t bytes, void* user);
agnes_status agnes_set_device_allocator(agnes_device_alloc_fn alloc, agnes_device_free_fn release, void* user);

/* Store options.
 *   AGNES_OPT_PROFILE: 1 = record HIP events around the phases of every
 *     hyperbatch (reported by agnes_batch_stats), 0 = off (default).
 *   AGNES_OPT_GATHER_GROUPS: most workgroups of the row-copy kernel, in
 *     [8, 2^22] (default 2^22); a launch never takes more workgroups than it
 *     has blocks of rows.  Fewer leave room for another stream's work.
 *   AGNES_OPT_GATHER_UNROLL: rows each lane group keeps in flight, 4, 8 or
 *     16; 0 (default) picks by row width: 16 for rows of 1 KiB up to 2 KiB
 *     (one 16-byte piece per lane), 4 for all others.
 *   AGNES_OPT_GATHER_NONTEMPORAL: 1 = write gathered rows with non-temporal
 *     stores (default), 0 = ordinary stores.
 *   AGNES_OPT_GATHER_CHUNKS: the row copy runs as this many consecutive
 *     launches over consecutive parts of the bucket, in [1, 64] (default 1);
 *     kernels of other streams are dispatched between them.
 *   AGNES_OPT_SAMPLING_GRAPH: 0 = every hyperbatch launches its sampling
 *     kernels one by one.  1 = a batch that begins two hyperbatches of the
 *     same shape in a row (same H, B, fanouts and store, and the same scratch
 *     buffers) captures the sampling kernels as a HIP graph and from then on
 *     replays it with one graph launch per hyperbatch; a batch holds one such
 *     graph and captures again when the shape changes.  2 (default) = as 1
 *     for shapes whose hops can sample at most 2^20 edges in all (H x frontier
 *     capacity x fanout, summed over the hops), as 0 for larger ones.  Replay
 *     shortens small, launch-bound hyperbatches but slows large hyperbatches
 *     that sample concurrently on several streams.
 *   AGNES_OPT_JOIN_PATH: how each hop unites the sampled neighbours with the
 *     nodes already held and relabels them.  0 (default): a device-wide radix
 *     sort of the sampled neighbours and a merge-path join with the list;
 *     1: node-range buckets, each joined in workgroup memory (a dense
 *     (node, minibatch) table for narrow buckets such as one hub, a sort in
 *     workgroup memory for the others).
 *   AGNES_OPT_BUCKET_CAP: old and new entries one sorted node-range bucket may
 *     hold, in [64, 2048] (default 2048).  A hyperbatch with a bucket above it
 *     is sampled again with the radix sort (same results); a smaller value
 *     only makes that happen more often.
 *   AGNES_OPT_SAMPLING_GROUPS: most workgroups of each sampling-phase kernel
 *     that loops over its work (the sampler, the radix passes, the join), in
 *     [256, 4096]; 0 (default) chooses per hop: the power of two at or below
 *     its bound of sampled edges (H x frontier capacity x fanout) / 32768,
 *     within [512, 2048].  4096
 *     leaves each kernel at its own limit, 2048 for most.  Fewer need fewer
 *     dispatch slots beside a running row copy of another hyperbatch, which
 *     holds most of them; a large hop needs more to hide its latency.
 * Options change launch shapes and store kinds only, never results. */
typedef enum {
    AGNES_OPT_PROFILE = 1,
    AGNES_OPT_GATHER_GROUPS = 2,
    AGNES_OPT_GATHER_UNROLL = 3,
    AGNES_OPT_GATHER_NONTEMPORAL = 4,
    AGNES_OPT_GATHER_CHUNKS = 5,
    AGNES_OPT_SAMPLING_GRAPH = 6,
    AGNES_OPT_JOIN_PATH = 7,
    AGNES_OPT_BUCKET_CAP = 8,
    AGNES_OPT_SAMPLING_GROUPS = 9
} agnes_option;
agnes_status agnes_store_set_option(agnes_store* store, agnes_option opt, int64_t value);

/* Staged feature tier (Sec. 3.4(1): blocks pinned in a buffer until the
 * current iteration has processed them, LRU replacement; Sec. 3.2(1): fixed-size
 * blocks as the unit of I/O).  Like agnes_build_blocks, but the feature
 * matrix is kept in library-owned pinned host memory (its padded copy:
 * ceil(num_nodes / rows_per_block) blocks) and only a pool of `pool_blocks`
 * feature-block slots (pool_blocks * rows_per_block * row_bytes bytes) is
 * allocated in HBM.  The topology stays in HBM.
 *
 * Every hyperbatch prepared on such a store needs the feature blocks that its
 * final bucket touches (ascending block ids).  They are taken in rounds of at
 * most pool_blocks blocks.  Within a round, the blocks already in the pool are
 * hits: each is used in turn (ascending) and so pinned for the round.  Then
 * each missing block (ascending) takes the lowest slot that never held a
 * block, or else the least recently used slot that is not pinned in this
 * round, and is used.  The GPU copies the missing blocks from host memory into
 * their slots, then copies the round's rows.  Slots keep their blocks across
 * hyperbatches, so a later hyperbatch hits blocks staged earlier.  Outputs are
 * identical to a store with HBM-resident features.
 * Hyperbatches of one store are gathered one at a time in the order their
 * finish calls are made (each waits for the previous gather on any stream).
 * agnes_batch_finish finds the needed blocks on the batch's begin stream and
 * waits on the host only for them, so the host plans a hyperbatch's rounds
 * while earlier hyperbatches still stage and gather (with a feature cache, the
 * search also waits for the previous hyperbatch's admissions).
 * Errors: as agnes_build_blocks; pool_blocks < 1 -> AGNES_ERR_INVALID. */
agnes_status agnes_build_blocks_staged(const agnes_csr* csr, const agnes_features* feat,
                                       uint64_t block_bytes, int64_t pool_blocks, void* hip_stream,
                                       agnes_store** out);

/* Staged tier with a feature cache (Sec. 3.4(2): the number of accesses to
 * every feature vector is counted, and vectors whose count reaches a
 * threshold are kept in a feature cache; the others are loaded with their
 * blocks when needed).  As agnes_build_blocks_staged, plus an HBM cache of
 * `cache_rows` feature rows (the cache index table maps a node to its cache
 * row):
 *   - a hyperbatch's rows found in the cache are copied from it; the needed
 *     feature blocks are the blocks of its other rows (staged and pooled as
 *     above);
 *   - after its gather, every row the hyperbatch gathered adds the number of
 *     its minibatches to its access count; rows not in the cache whose count
 *     is now >= `threshold` enter it, ascending by node id, while it has room
 *     (copied from host memory); rows never leave it.
 * cache_rows = 0 gives agnes_build_blocks_staged.  Errors: pool_blocks < 1,
 * cache_rows < 0 or threshold < 1 -> AGNES_ERR_INVALID. */
agnes_status agnes_build_blocks_cached(const agnes_csr* csr, const agnes_features* feat,
                                       uint64_t block_bytes, int64_t pool_blocks, int64_t cache_rows,
                                       int64_t threshold, void* hip_stream, agnes_store** out);

/* Feature-tier counters of a prepared hyperbatch (all zero for a store with
 * HBM-resident features): needed feature blocks (the blocks of its rows not in
 * the feature cache; = agnes_stats.feat_blocks without a cache), blocks copied
 * from host memory, blocks found in the pool, rounds, bytes copied from host
 * memory for blocks, distinct rows served by the feature cache, rows that
 * entered the cache after this hyperbatch, rows in the cache after it, and the
 * device time of the gather including staging and admission when profiling is
 * on (else -1). */
typedef struct {
    int64_t needed_blocks;
    int64_t staged_blocks;
    int64_t hit_blocks;
    int64_t rounds;
    int64_t staged_bytes;
    int64_t cache_hit_rows;
    int64_t admitted_rows;
    int64_t cached_rows;
    float gather_ms;
} agnes_tier_stats;

agnes_status agnes_batch_tier_stats(const agnes_batch* batch, agnes_tier_stats* out);  /* waits for the batch */

/* GraphSAGE forward pass over a prepared hyperbatch (the step after data
 * preparation; Eq. (1), Sec. 3.1): L layers, layer i on hop l = L-1-i, from the
 * outermost hop to the targets.  For every destination node v of hop l in
 * minibatch j (local ids 0 .. layer_sizes[j][l]-1):
 *   m_v = mean of h_u over the sampled neighbours u of v (zero vector when v
 *         has none), with h the layer's input embeddings (layer 0: the
 *         gathered feature rows, converted to float);
 *   z_v = W_i [h_v ; m_v] + b_i,   h'_v = max(z_v, 0) for i < L-1, z_v for the last layer.
 * Node v's own input row is the same local id of the previous node set (the
 * destination nodes of a hop are a prefix of its source nodes).
 *   dims[0] = feature dim; dims[i+1] = output dim of layer i; every dims[i]
 *     must be a positive multiple of 32, at most 4096.
 *   weight[i]: device bf16 (raw uint16 bits), [dims[i+1]][2*dims[i]] row-major:
 *     columns 0 .. dims[i]-1 multiply h_v, the others m_v (the layout of a
 *     linear layer's weight, output-major); 16-byte aligned.
 *   bias[i]: device float32 [dims[i+1]].
 *   out: device float32 [H*B][dims[L]]: the targets' embeddings, minibatch-major
 *     in the order the targets were given; 16-byte aligned.
 * Arithmetic: m_v is accumulated in float32; [h_v ; m_v] is rounded to bf16
 * and multiplied with bf16 MFMA, accumulating in float32; hidden embeddings
 * are stored as bf16.  The call enqueues on hip_stream after the batch's
 * gather and returns; the batch owns the intermediate buffers.
 * Errors: a batch without a finished hyperbatch, L != the batch's hop count,
 * dims out of range, dims[0] != the feature dim, a NULL or misaligned pointer
 * -> AGNES_ERR_INVALID. */
typedef struct {
    int32_t L;
    int32_t dims[AGNES_MAX_LAYERS + 1];
    const uint16_t* weight[AGNES_MAX_LAYERS];
    const float* bias[AGNES_MAX_LAYERS];
} agnes_sage_model;

agnes_status agnes_sage_forward(agnes_batch* batch, const agnes_sage_model* model, float* out,
                                void* hip_stream);

/* The same forward for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): it
 * calls no hipMalloc, hipFree or other allocating routine.  Same arguments,
 * checks, kernels and results as agnes_sage_forward.  Its intermediate rows
 * (the per-layer offsets, the [h_v ; m_v] rows and the hidden embeddings) live
 * in one static device array of AGNES_NOALLOC_SCRATCH_BYTES per GPU, held
 * from the first call on that GPU until the process ends; a forward needing
 * more (bytes: 8 * 4 * L * (H+1) + 2 * max_i(M_i * 2 * dims[i]) + 4 *
 * max_{i<L-1}(M_i * dims[i+1]), each rounded up to 256, with M_i the
 * destination rows of layer i over the hyperbatch) fails with
 * AGNES_ERR_RANGE before anything is enqueued.  Every call on one GPU uses
 * that GPU's single array: calls whose work overlaps on one GPU (several
 * streams, or several host threads) race and must be serialised by the
 * caller, e.g. by enqueueing them on one stream.  The next hyperbatch begun on
 * the batch waits for the forward, as with agnes_sage_forward. */
#define AGNES_NOALLOC_SCRATCH_BYTES (64ull << 20)
agnes_status agnes_sage_forward_noalloc(agnes_batch* batch, const agnes_sage_model* model, float* out,
                                        void* hip_stream);

/* Store facts: out[0] num_nodes, out[1] num_edges, out[2] topology blocks,
 * out[3] edges per topology block, out[4] feature blocks, out[5] rows per
 * feature block, out[6] row_bytes, out[7] device bytes held by the store. */
agnes_status agnes_store_info(const agnes_store* store, int64_t out[8]);

/* Object index table (Sec. 3.2(2)): copies to host first_node[b] and
 * last_node[b] (int32, -1 for a block that no object starts in) for every
 * topology block b; each array needs agnes_store_info()[2] entries. */
agnes_status agnes_store_object_table(const agnes_store* store, int32_t* first_node,
                                      int32_t* last_node);

/* Release a store or a batch (NULL is a no-op; a batch's enqueued work is
 * waited for).  A store must outlive the work of its batches. */
void agnes_free(void* handle);

/* Message of the last failure on the calling thread ("" if none); valid until
 * the next call on that thread. */
const char* agnes_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* AGNES_H */
