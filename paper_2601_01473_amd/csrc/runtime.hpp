// Host runtime types of the library: error state, device buffers, the block
// store, the per-store scratch workspace and the batch (outputs of a prepare).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <climits>
#include <deque>
#include <string>
#include <utility>
#include <vector>

#include "../../include/agnes.h"

namespace agnes {

// ----------------------------------------------------------------- errors

struct Error {
    agnes_status code;
    std::string msg;
};

void set_last_error(const std::string& msg);
void clear_last_error();

#define AGNES_CHECK_HIP(expr)                                                               \
    do {                                                                                    \
        hipError_t e_ = (expr);                                                             \
        if (e_ != hipSuccess)                                                               \
            throw ::agnes::Error{e_ == hipErrorOutOfMemory ? AGNES_ERR_NOMEM : AGNES_ERR_DEVICE, \
                                 std::string(#expr) + ": " + hipGetErrorString(e_)};        \
    } while (0)

#define AGNES_REQUIRE(cond, code, msg)                                                      \
    do {                                                                                    \
        if (!(cond)) throw ::agnes::Error{(code), (msg)};                                   \
    } while (0)

// Debug mode: with AGNES_DEBUG_SYNC=1 in the environment when the library is
// loaded, every kernel launch is followed by a synchronisation of its stream
// (skipped while the stream is being captured into a graph) and an error check,
// so a failing kernel is reported under the name of the launch that enqueued it.
bool debug_sync();
void check_launch(hipStream_t st, const char* what);

#define AGNES_LAUNCH(kernel, grid, block, lds, st, ...)                                    \
    do {                                                                                    \
        hipLaunchKernelGGL(kernel, grid, block, lds, st, __VA_ARGS__);                      \
        ::agnes::check_launch((st), #kernel);                                               \
    } while (0)

// Host-side ranges around the library's phases (roctx; seen by rocprofv3
// --marker-trace, free when no profiler is attached).
struct Range {
    explicit Range(const char* name);
    ~Range();
    Range(const Range&) = delete;
    Range& operator=(const Range&) = delete;
};

// ----------------------------------------------------------------- device buffer

// The process-wide device allocator: hipMalloc / hipFree unless the caller
// installed callbacks (agnes_set_device_allocator).
struct DeviceAllocator {
    agnes_device_alloc_fn alloc = nullptr;
    agnes_device_free_fn release = nullptr;
    void* user = nullptr;
};
DeviceAllocator& device_allocator();

// An owned device allocation that only grows (contents are not preserved).
// A buffer from the caller's allocator remembers the free callback that pairs
// with it and its device; before handing the memory back it waits for that
// device's enqueued work, as hipFree does, since a caching allocator may give
// the block to its next user at once.
struct DevBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
    agnes_device_free_fn free_fn = nullptr;   // null: the memory came from hipMalloc
    void* free_user = nullptr;
    int device = 0;
    ~DevBuf() { release(); }
    void release() {
        if (ptr) {
            if (free_fn) {
                int cur = 0;
                if (hipGetDevice(&cur) == hipSuccess && cur != device) (void)hipSetDevice(device);
                (void)hipDeviceSynchronize();
                free_fn(ptr, (uint64_t)bytes, free_user);
                if (cur != device) (void)hipSetDevice(cur);
            } else {
                (void)hipFree(ptr);
            }
        }
        ptr = nullptr;
        bytes = 0;
        free_fn = nullptr;
        free_user = nullptr;
    }
    // Make room for `need` bytes; returns true when a new allocation was made.
    bool reserve(size_t need) {
        if (need <= bytes && ptr) return false;
        release();
        size_t b = need ? need : 256;
        const DeviceAllocator& a = device_allocator();
        if (a.alloc) {
            void* p = a.alloc((uint64_t)b, a.user);
            if (!p) throw Error{AGNES_ERR_NOMEM, "the device allocator returned no memory for " + std::to_string(b) + " bytes"};
            if ((uintptr_t)p & 255u) {
                a.release(p, (uint64_t)b, a.user);
                throw Error{AGNES_ERR_INVALID, "the device allocator must return 256-byte aligned memory"};
            }
            AGNES_CHECK_HIP(hipGetDevice(&device));
            ptr = p;
            free_fn = a.release;
            free_user = a.user;
        } else {
            AGNES_CHECK_HIP(hipMalloc(&ptr, b));
        }
        bytes = b;
        return true;
    }
    // Same, with 25% headroom when growing, for sizes that vary call to call.
    bool reserve_slack(size_t need) {
        if (need <= bytes && ptr) return false;
        return reserve(need + need / 4);
    }
    template <typename T> T* as() const { return static_cast<T*>(ptr); }
};

// Pinned host memory that only grows.
struct PinnedBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
    ~PinnedBuf() {
        if (ptr) (void)hipHostFree(ptr);
    }
    // Same, with 25% headroom when growing, for sizes that vary call to call.
    void reserve_slack(size_t need) {
        if (need <= bytes && ptr) return;
        reserve(need + need / 4);
    }
    void reserve(size_t need) {
        if (need <= bytes && ptr) return;
        if (ptr) (void)hipHostFree(ptr);
        ptr = nullptr;
        bytes = 0;
        AGNES_CHECK_HIP(hipHostMalloc(&ptr, need ? need : 256, hipHostMallocDefault));
        bytes = need ? need : 256;
    }
};

constexpr uint32_t kStoreMagic = 0x53454E47u;   // "GNES"
constexpr uint32_t kBatchMagic = 0x42454E47u;

// Counters and statistics kept in device memory during a prepare.
struct Ctl {
    int64_t R;          // requests of the current hop
    int64_t S;          // sampled edges of the current hop
    int64_t n_new;      // new nodes of the current hop (all minibatches)
    int64_t rows;       // gathered rows (sum of |N_j|)
    int64_t err;        // bit 0: target out of range, bit 1: duplicate target, bit 2: capacity
    int64_t targets;    // H * B
    int64_t tier_unc;   // staged tier: list entries whose rows are not in the feature cache
    int64_t tier_nb;    // staged tier: needed feature blocks
    int64_t tier_hits;  // staged tier: distinct rows served by the feature cache
    int64_t tier_cand;  // staged tier: rows that reached the threshold this hyperbatch
    int64_t tier_admitted, tier_cached;
    int64_t requests[AGNES_MAX_LAYERS];
    int64_t sampled[AGNES_MAX_LAYERS];
    int64_t new_nodes[AGNES_MAX_LAYERS];
    int64_t topo_blocks[AGNES_MAX_LAYERS];
};

// Scratch memory of a prepare, owned by the store and grown on demand.
struct Workspace {
    DevBuf nodes;                     // [H][capN] node lists in local-id order
    DevBuf size, newcnt;              // per minibatch
    DevBuf req_off, mb_off;           // [H+1] int64
    DevBuf sync;                      // Ctl, layer sizes, edge counts (read by the host)
    PinnedBuf sync_host;
    DevBuf cnt, e_off;                // per request
    DevBuf rl_key[2], rl_val[2];      // (node, minibatch) list and local ids, two buffers
    DevBuf skey, sval, skey2, sval2;  // sort buffers (sampled neighbours, targets)
    DevBuf split;                     // join: list entries before every tile boundary
    DevBuf ghist, gemit;              // join: per group new nodes per minibatch, merged entries
    DevBuf rs_hist, rs_dtot;          // radix-sort histograms
    DevBuf scan_part;                 // scan partial sums
    DevBuf topo_part;                 // per sampler workgroup: Bck rows it opened
    DevBuf acoff;                     // node-range buckets: old list entries before each coarse bucket
    DevBuf params;                    // per-call values the sampling kernels read (targets, seed, minibatch base)
    DevBuf targets;                   // targets uploaded from host memory by the call
    PinnedBuf targets_host;           // their pinned staging copy
    DevBuf blk_flag, blk_off;         // staged tier: flags over the final list and their offsets
    DevBuf unc;                       // staged tier: list entries whose rows are not in the feature cache
    DevBuf need;                      // staged tier: [needed blocks] first list entry, then block ids
    DevBuf plan;                      // staged tier: the rounds' (block, slot) updates and misses
    PinnedBuf need_host, plan_host;
    size_t plan_used = 0;             // staged tier: bytes of the current plan
    hipEvent_t ev[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
};

struct Store {
    uint32_t magic = kStoreMagic;
    int device = 0;
    int max_lds = 65536;              // LDS bytes one workgroup may use on the device
    int64_t num_nodes = 0, num_edges = 0;
    int offsets64 = 0;                // 1: int64 offsets, 0: int32
    int64_t e_blk = 0;                // edges per topology block
    int e_blk_log2 = 0;
    int64_t nblk = 0;                 // topology blocks
    int64_t row_bytes = 0;
    int feat_dtype = AGNES_FLOAT32;   // element type of the feature rows
    int64_t rpb = 0;                  // feature rows per block
    int64_t nfblk = 0;                // feature blocks
    int64_t block_bytes = 0;
    int64_t max_degree = 0;
    int node_bits = 0;                // bits of a node id (ceil log2 num_nodes)
    DevBuf offsets, indices, features, first_node, last_node;
    // Node-range buckets of the join (bucket.hip): nlev nested levels, finest
    // first; lev_info_host / lev_info: [nlev][2] (offset of the level's
    // boundaries in bnd, bucket count); bnd: every level's boundaries
    // (count + 1 ascending node ids from 0 to num_nodes).
    int nlev = 0;
    std::vector<int32_t> lev_info_host;
    DevBuf bnd, lev_info;
    int join_path = 0;                // 1 = node-range buckets, 0 = radix sort and merge-path join (default)
    int bucket_cap = 2048;            // entries of a sorted sub-bucket (at most kBucketCap)
    int sample_groups = 0;            // most workgroups of a sampling-phase kernel that loops over its
                                      // work; 0 = chosen per hop by its size
    // Staged feature tier (features in pinned host memory, an HBM pool of
    // feature-block slots).  Not used when tiered == 0 (features in HBM).
    // The pool's host-side bookkeeping changes with every planned hyperbatch.
    int tiered = 0;
    void* host_feat = nullptr;        // pinned host copy of the padded feature matrix
    void* host_feat_dev = nullptr;    // its device-visible address
    int64_t pool_blocks = 0;          // slots of the pool (rpb rows each)
    int64_t pool_rows = 0;            // pool_blocks * rpb: the feature cache's rows follow them in `pool`
    int64_t cache_rows = 0;           // rows of the feature cache (0: none)
    int64_t cache_threshold = 1;      // access count at which a row enters the cache
    DevBuf pool;                      // [pool_blocks * rpb + cache_rows][row_bytes]
    DevBuf tch;                       // [num_nodes] int32: cache row of node u, or -1
    DevBuf acc_count;                 // [num_nodes] uint32: accesses of node u's feature row so far
    DevBuf cache_used;                // int64: rows in the cache
    DevBuf tbuf;                      // [nfblk] int32: slot holding feature block b, or -1
    mutable std::vector<int32_t> slot_block;  // host view of the pool: block in slot s, or -1
    mutable std::vector<int64_t> slot_stamp;  // access number of slot s's last use (-1: never)
    mutable std::vector<int32_t> block_slot;  // host mirror of tbuf
    // Replacement order: (access number, slot) in access order; an entry whose
    // slot was used again later is stale and skipped.
    mutable std::deque<std::pair<int64_t, int32_t>> lru;
    mutable int64_t accesses = 0;     // pool accesses so far (hits and stagings)
    mutable int64_t next_free = 0;    // lowest never-used slot
    mutable int64_t tier_clock = 0;   // rounds planned so far
    hipEvent_t pool_free = nullptr;   // the last enqueued tiered gather is done with the pool
    ~Store() {
        if (host_feat) (void)hipHostFree(host_feat);
        if (pool_free) (void)hipEventDestroy(pool_free);
    }
    int profile = 0;
    int sampling_graph = 2;           // 1 = replay the sampling kernels from a captured HIP graph, 0 = never,
                                      // 2 = for hyperbatches of at most kGraphAutoEdges sampled edges
    int gather_groups = 1 << 22;      // workgroups of the row-copy kernel (upper bound)
    int gather_unroll = 0;            // rows in flight per lane group (4, 8 or 16; 0 = by row width)
    int gather_nt = 1;                // 1 = non-temporal stores of the gathered rows
    int gather_chunks = 1;            // consecutive launches the row copy is split into
};

// A batch: the outputs of one hyperbatch and the scratch memory that produces
// them.  State: kIdle -> (begin) kSampled -> (finish) kGathering -> (wait) kDone.
enum BatchState { kIdle = 0, kSampled = 1, kGathering = 2, kDone = 3 };

struct Batch {
    uint32_t magic = kBatchMagic;
    const Store* store = nullptr;
    int32_t H = 0, B = 0, L = 0;
    int state = kIdle;
    hipStream_t stream = nullptr;     // stream of the sampling phase
    hipEvent_t sampled = nullptr;     // sizes of the outputs are in ws.sync_host
    hipEvent_t gathered = nullptr;    // outputs and statistics are complete
    // The events that mark those points for the current hyperbatch: `sampled`
    // and `gathered`, or, when it is profiled, the timing events recorded at
    // the same points (one marker fewer per phase on the stream).
    int prof = 0;
    hipEvent_t sampled_at = nullptr, gathered_at = nullptr;
    hipEvent_t needed = nullptr;      // staged tier: the needed feature blocks are in ws.need_host
    int64_t capN = 0;
    int64_t rows_max = 0;             // node-list capacity of the hyperbatch (sizes the sync block)
    int cur = 0;                      // which list buffer holds the final list
    // The sampling phase wrote the output node ids (nodes) itself (radix-sort
    // path); otherwise the row copy writes them.
    bool ids_in_chain = false;
    // The begun hyperbatch's arguments, for sampling it again on the radix-sort
    // path when a node-range bucket overflows (fallbacks counts those).
    std::vector<int32_t> fanouts;
    uint64_t seed = 0;
    int64_t mb_base = 0;
    const int32_t* targets_dev = nullptr;
    int64_t fallbacks = 0;
    int64_t need_cap = 0;             // staged tier: entries of each array in ws.need
    std::vector<int64_t> node_off;
    std::vector<int32_t> layer_sizes;
    std::vector<int64_t> rp_off[AGNES_MAX_LAYERS];
    std::vector<int64_t> col_off[AGNES_MAX_LAYERS];
    DevBuf nodes, features;
    DevBuf row_ptr[AGNES_MAX_LAYERS], col[AGNES_MAX_LAYERS];
    Workspace ws;
    agnes_stats stats{};
    agnes_tier_stats tier{};
    // GraphSAGE forward (sage.hip): per-layer offsets, the [h ; mean] rows, hidden embeddings
    PinnedBuf sage_host;
    DevBuf sage_off, sage_a, sage_h[2];
    hipEvent_t sage_ev = nullptr;     // the offsets upload has left sage_host
    // The end of the last forward enqueued on this batch: the next hyperbatch
    // and the next forward wait for it before they overwrite what it reads.
    hipEvent_t sage_done = nullptr;
    bool sage_pending = false;
    // Device copies of the layer sizes [H][L+1] and per-hop edge counts [H][L]
    // (inside ws.sync), valid once the hyperbatch's sampling has finished.
    const int32_t* d_lsz = nullptr;
    const int64_t* d_ecount = nullptr;
    // The sampling kernels of one hyperbatch shape, captured as a HIP graph.
    // chain_key lists everything the captured launches depend on (shape, store,
    // buffer addresses); a call with another key runs kernel by kernel and is
    // captured when the next call repeats its key.
    hipGraphExec_t chain = nullptr;
    hipStream_t cap_stream = nullptr; // private stream the chain is captured on (never runs work)
    std::vector<uint64_t> chain_key, last_key;
    ~Batch() {
        if (chain) (void)hipGraphExecDestroy(chain);
        if (cap_stream) (void)hipStreamDestroy(cap_stream);
        if (sampled) (void)hipEventDestroy(sampled);
        if (gathered) (void)hipEventDestroy(gathered);
        if (needed) (void)hipEventDestroy(needed);
        if (sage_ev) (void)hipEventDestroy(sage_ev);
        if (sage_done) (void)hipEventDestroy(sage_done);
        for (auto& e : ws.ev)
            if (e) (void)hipEventDestroy(e);
    }
};

// Pipeline entry points (pipeline.hip).  begin enqueues the sampling hops on
// `stream` and returns; finish waits for the output sizes, makes room for the
// outputs and enqueues the gather on `stream`; wait blocks until the batch is
// complete and fills its statistics.
// targets_on_host: targets is host memory, copied by the call (through pinned
// memory) to the device on `stream`; otherwise it is device memory.
void begin_hyperbatch(const Store& s, Batch& b, const int32_t* targets, bool targets_on_host, int32_t H,
                      int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                      hipStream_t stream);
void finish_hyperbatch(Batch& b, hipStream_t stream);
void wait_batch(Batch& b);
// GraphSAGE forward over a prepared batch (sage.hip); enqueues on `stream`.
void sage_forward(Batch& b, const agnes_sage_model& m, float* out, hipStream_t stream);
// The same without any allocation: scratch space from a static device array
// of kNoAllocScratchBytes per GPU (sage.hip).
constexpr size_t kNoAllocScratchBytes = AGNES_NOALLOC_SCRATCH_BYTES;
void sage_forward_noalloc(Batch& b, const agnes_sage_model& m, float* out, hipStream_t stream);
// Store construction (store.hip).
// pool_blocks == 0: features in HBM; > 0: staged feature tier with that many
// slots and a feature cache of cache_rows rows (0: none).
Store* build_store(const agnes_csr* csr, const agnes_features* feat, uint64_t block_bytes,
                   int64_t pool_blocks, int64_t cache_rows, int64_t cache_threshold, hipStream_t stream);

// ----------------------------------------------------------------- primitives (prims.hip)

// Exclusive scan of n int32 counts (n read from *n_dev, at most n_max) into
// out[0..n] int64; out[n] = total, also stored to *total_dev when not null.  When
// `nonzero` is not null, the number of nonzero inputs is added to *nonzero.
void scan_counts(const int32_t* in, int64_t* out, const int64_t* n_dev, int64_t n_max,
                 int64_t* total_dev, int64_t* partials, hipStream_t st, int64_t* nonzero = nullptr);
// Partial sums a scan needs (the size of `partials`).
int64_t scan_partials_needed();
// Workgroups (ranges) of a scan over at most n_max elements, and its final
// pass alone, for a reduce pass fused into the kernel that produces the counts
// (it must write partials[g] = the sum of range g, as scan_range splits them).
// The final pass writes 32-bit offsets: the caller guarantees a total below
// 2^32 (a hop's edge numbers, by the plan's bound); *total_dev is 64-bit.
int scan_groups(int64_t n_max);
void scan_counts_final(const int32_t* in, uint32_t* out, const int64_t* n_dev, int64_t n_max, int64_t* total_dev,
                       const int64_t* partials, hipStream_t st);

// Stable LSD radix sort of 32-bit keys with 32-bit values on key bits
// [0, bits), in the fewest passes of 8-10-bit digits; n read from *n_dev (at
// most n_max).  With
// vals_iota the input values are 0, 1, 2, ... (vals is then only an output
// buffer).  hist needs radix_hist_entries(n_max) entries, dtot
// radix_dtot_entries().  Returns 0 when the result is in keys/vals and 1 when it
// is in keys_tmp/vals_tmp.
// max_groups caps the workgroups of the histogram and scatter kernels (they
// loop over the tiles).
int radix_sort_pairs32(uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                       const int64_t* n_dev, int64_t n_max, int bits, uint32_t* hist,
                       uint32_t* dtot, hipStream_t st, bool vals_iota = false, int max_groups = 2048);
int64_t radix_hist_entries(int64_t n_max);
// Keys per thread (8 or 16) and tiles of a radix pass over at most n_max keys.
int radix_items(int64_t n_max);
int64_t radix_tiles(int64_t n_max);
int64_t radix_dtot_entries();

// Philox4x64-10 words of n (counter [4], key [2]) pairs, device arrays (prims.hip).
void philox_words(const uint64_t* counters, const uint64_t* keys, int64_t n, uint64_t* out, hipStream_t st);

// Fill n 32-bit words with a value (a kernel, so that it can be captured in a graph).
void fill_u32(void* p, uint32_t value, int64_t n, hipStream_t st);

inline int grid_for(int64_t n, int max_blocks = 4096) {
    int64_t g = (n + 255) / 256;
    if (g < 1) g = 1;
    if (g > max_blocks) g = max_blocks;
    return (int)g;
}

}  // namespace agnes
