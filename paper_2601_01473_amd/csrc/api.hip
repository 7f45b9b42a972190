// The C ABI (include/agnes.h): argument checks, error mapping and handle
// management around the store (store.hip) and the pipeline (pipeline.hip).
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "bucket.hpp"
#include "runtime.hpp"

namespace agnes {

static thread_local std::string g_last_error;

DeviceAllocator& device_allocator() {
    static DeviceAllocator a;
    return a;
}

void set_last_error(const std::string& msg) { g_last_error = msg; }
void clear_last_error() { g_last_error.clear(); }

bool debug_sync() {
    static const bool on = [] {
        const char* v = std::getenv("AGNES_DEBUG_SYNC");
        return v && v[0] && std::strcmp(v, "0") != 0;
    }();
    return on;
}

void check_launch(hipStream_t st, const char* what) {
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && debug_sync()) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(st, &cs) == hipSuccess && cs == hipStreamCaptureStatusNone) {
            e = hipStreamSynchronize(st);
            if (e == hipSuccess) e = hipGetLastError();
        }
    }
    if (e != hipSuccess)
        throw Error{e == hipErrorOutOfMemory ? AGNES_ERR_NOMEM : AGNES_ERR_DEVICE,
                    std::string("kernel ") + what + ": " + hipGetErrorString(e)};
}

Range::Range(const char* name) { (void)roctxRangePushA(name); }
Range::~Range() { (void)roctxRangePop(); }

template <typename F>
static agnes_status guarded(F&& f) {
    try {
        clear_last_error();
        f();
        return AGNES_OK;
    } catch (const Error& e) {
        set_last_error(e.msg);
        return e.code;
    } catch (const std::bad_alloc&) {
        set_last_error("host allocation failed");
        return AGNES_ERR_NOMEM;
    } catch (const std::exception& e) {
        set_last_error(e.what());
        return AGNES_ERR_INTERNAL;
    } catch (...) {
        set_last_error("unknown internal error");
        return AGNES_ERR_INTERNAL;
    }
}

static Store* as_store(void* p) {
    Store* s = static_cast<Store*>(p);
    AGNES_REQUIRE(s && s->magic == kStoreMagic, AGNES_ERR_INVALID, "not a store handle");
    return s;
}

}  // namespace agnes

using namespace agnes;

extern "C" {

agnes_status agnes_build_blocks(const agnes_csr* csr, const agnes_features* feat,
                                uint64_t block_bytes, void* hip_stream, agnes_store** out) {
    if (out) *out = nullptr;
    return guarded([&] {
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        Store* s = build_store(csr, feat, block_bytes, 0, 0, 1, (hipStream_t)hip_stream);
        *out = reinterpret_cast<agnes_store*>(s);
    });
}

agnes_status agnes_build_blocks_staged(const agnes_csr* csr, const agnes_features* feat,
                                       uint64_t block_bytes, int64_t pool_blocks, void* hip_stream,
                                       agnes_store** out) {
    if (out) *out = nullptr;
    return guarded([&] {
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        AGNES_REQUIRE(pool_blocks >= 1, AGNES_ERR_INVALID, "pool_blocks must be >= 1");
        Store* s = build_store(csr, feat, block_bytes, pool_blocks, 0, 1, (hipStream_t)hip_stream);
        *out = reinterpret_cast<agnes_store*>(s);
    });
}

agnes_status agnes_build_blocks_cached(const agnes_csr* csr, const agnes_features* feat,
                                       uint64_t block_bytes, int64_t pool_blocks, int64_t cache_rows,
                                       int64_t threshold, void* hip_stream, agnes_store** out) {
    if (out) *out = nullptr;
    return guarded([&] {
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        AGNES_REQUIRE(pool_blocks >= 1, AGNES_ERR_INVALID, "pool_blocks must be >= 1");
        AGNES_REQUIRE(cache_rows >= 0, AGNES_ERR_INVALID, "cache_rows must not be negative");
        AGNES_REQUIRE(threshold >= 1, AGNES_ERR_INVALID, "threshold must be >= 1");
        AGNES_REQUIRE(cache_rows < 0x7FFFFFFFll, AGNES_ERR_INVALID, "cache_rows must be < 2^31");
        Store* s = build_store(csr, feat, block_bytes, pool_blocks, cache_rows, threshold, (hipStream_t)hip_stream);
        *out = reinterpret_cast<agnes_store*>(s);
    });
}

}  // extern "C"

namespace agnes {

// Argument checks shared by prepare and begin; returns the batch to fill (the
// one passed in, or a new one).
static Batch* check_begin(agnes_store* store, const int32_t* targets, int32_t H, int32_t B,
                          const int32_t* fanouts, int32_t L, int64_t mb_base, Batch* reuse, Store*& s) {
    s = as_store(store);
    AGNES_REQUIRE(!reuse || (reuse->magic == kBatchMagic && reuse->store == s), AGNES_ERR_INVALID,
                  "the batch passed in was not produced by this store");
    AGNES_REQUIRE(targets, AGNES_ERR_INVALID, "targets must not be NULL");
    AGNES_REQUIRE(H >= 1 && H <= 4096, AGNES_ERR_INVALID, "H must be in [1, 4096]");
    AGNES_REQUIRE(B >= 1, AGNES_ERR_INVALID, "B must be >= 1");
    AGNES_REQUIRE((int64_t)H * B < 0x7FFFFFFFll, AGNES_ERR_RANGE, "H * B must be < 2^31");
    AGNES_REQUIRE(L >= 1 && L <= AGNES_MAX_LAYERS, AGNES_ERR_INVALID, "L must be in [1, 8]");
    AGNES_REQUIRE(fanouts, AGNES_ERR_INVALID, "fanouts must not be NULL");
    for (int l = 0; l < L; l++)
        AGNES_REQUIRE(fanouts[l] >= 0 && fanouts[l] <= 1024, AGNES_ERR_INVALID, "fanouts must be in [0, 1024]");
    AGNES_REQUIRE(mb_base >= 0, AGNES_ERR_INVALID, "mb_base must be >= 0");
    int dev = 0;
    AGNES_CHECK_HIP(hipGetDevice(&dev));
    AGNES_REQUIRE(dev == s->device, AGNES_ERR_INVALID, "the current device is not the store's device");
    return reuse ? reuse : new Batch();
}

static void release_batch(Batch* b) {
    if (b && b->magic == kBatchMagic) {
        if (b->state == kSampled || b->state == kGathering) {
            // let enqueued work finish before the memory goes away
            if (b->state == kSampled && b->sampled_at) (void)hipEventSynchronize(b->sampled_at);
            if (b->state == kGathering && b->gathered_at) (void)hipEventSynchronize(b->gathered_at);
        }
        if (b->sage_pending && b->sage_done) (void)hipEventSynchronize(b->sage_done);
        b->magic = 0;
        delete b;
    }
}

static Batch* as_batch(void* p) {
    Batch* b = static_cast<Batch*>(p);
    AGNES_REQUIRE(b && b->magic == kBatchMagic, AGNES_ERR_INVALID, "not a batch handle");
    return b;
}

}  // namespace agnes

extern "C" {

static agnes_status prepare_impl(agnes_store* store, const int32_t* targets, bool on_host, int32_t H, int32_t B,
                                 const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                                 void* hip_stream, agnes_batch** out) {
    Batch* reuse = (out && *out) ? reinterpret_cast<Batch*>(*out) : nullptr;
    if (out) *out = nullptr;
    Batch* b = nullptr;
    agnes_status rc = guarded([&] {
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        Store* s = nullptr;
        b = check_begin(store, targets, H, B, fanouts, L, mb_base, reuse, s);
        hipStream_t st = (hipStream_t)hip_stream;
        begin_hyperbatch(*s, *b, targets, on_host, H, B, fanouts, L, seed, mb_base, st);
        finish_hyperbatch(*b, st);
        wait_batch(*b);
        *out = reinterpret_cast<agnes_batch*>(b);
    });
    if (rc != AGNES_OK) release_batch(b ? b : reuse);
    return rc;
}

static agnes_status begin_impl(agnes_store* store, const int32_t* targets, bool on_host, int32_t H, int32_t B,
                               const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                               void* hip_stream, agnes_batch** out) {
    Batch* reuse = (out && *out) ? reinterpret_cast<Batch*>(*out) : nullptr;
    if (out) *out = nullptr;
    Batch* b = nullptr;
    agnes_status rc = guarded([&] {
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        Store* s = nullptr;
        b = check_begin(store, targets, H, B, fanouts, L, mb_base, reuse, s);
        begin_hyperbatch(*s, *b, targets, on_host, H, B, fanouts, L, seed, mb_base, (hipStream_t)hip_stream);
        *out = reinterpret_cast<agnes_batch*>(b);
    });
    if (rc != AGNES_OK) release_batch(b ? b : reuse);
    return rc;
}

agnes_status agnes_hyperbatch_prepare(agnes_store* store, const int32_t* targets, int32_t H,
                                      int32_t B, const int32_t* fanouts, int32_t L,
                                      uint64_t seed, int64_t mb_base, void* hip_stream,
                                      agnes_batch** out) {
    return prepare_impl(store, targets, true, H, B, fanouts, L, seed, mb_base, hip_stream, out);
}

agnes_status agnes_hyperbatch_prepare_device(agnes_store* store, const int32_t* targets, int32_t H,
                                             int32_t B, const int32_t* fanouts, int32_t L,
                                             uint64_t seed, int64_t mb_base, void* hip_stream,
                                             agnes_batch** out) {
    return prepare_impl(store, targets, false, H, B, fanouts, L, seed, mb_base, hip_stream, out);
}

agnes_status agnes_hyperbatch_begin(agnes_store* store, const int32_t* targets, int32_t H,
                                    int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed,
                                    int64_t mb_base, void* hip_stream, agnes_batch** out) {
    return begin_impl(store, targets, true, H, B, fanouts, L, seed, mb_base, hip_stream, out);
}

agnes_status agnes_hyperbatch_begin_device(agnes_store* store, const int32_t* targets, int32_t H,
                                           int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed,
                                           int64_t mb_base, void* hip_stream, agnes_batch** out) {
    return begin_impl(store, targets, false, H, B, fanouts, L, seed, mb_base, hip_stream, out);
}

agnes_status agnes_batch_finish(agnes_batch* batch, void* hip_stream) {
    Batch* b = nullptr;
    agnes_status rc = guarded([&] {
        b = as_batch(batch);
        finish_hyperbatch(*b, (hipStream_t)hip_stream);
    });
    return rc;
}

agnes_status agnes_batch_wait(agnes_batch* batch) {
    return guarded([&] { wait_batch(*as_batch(batch)); });
}

agnes_status agnes_batch_view_get(const agnes_batch* batch, agnes_batch_view* out) {
    return guarded([&] {
        const Batch* b = as_batch((void*)batch);
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        AGNES_REQUIRE(b->state == kGathering || b->state == kDone, AGNES_ERR_INVALID,
                      "the batch holds no finished hyperbatch");
        memset(out, 0, sizeof(*out));
        out->H = b->H;
        out->L = b->L;
        out->row_bytes = b->store->row_bytes;
        out->node_off = b->node_off.data();
        out->layer_sizes = b->layer_sizes.data();
        out->nodes = b->nodes.as<int32_t>();
        for (int l = 0; l < b->L; l++) {
            out->rp_off[l] = b->rp_off[l].data();
            out->row_ptr[l] = b->row_ptr[l].as<int32_t>();
            out->col_off[l] = b->col_off[l].data();
            out->col[l] = b->col[l].as<int32_t>();
        }
        out->features = b->features.ptr;
    });
}

agnes_status agnes_batch_stats(const agnes_batch* batch, agnes_stats* out) {
    return guarded([&] {
        Batch* b = as_batch((void*)batch);
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        wait_batch(*b);
        *out = b->stats;
    });
}

agnes_status agnes_sage_forward(agnes_batch* batch, const agnes_sage_model* model, float* out,
                                void* hip_stream) {
    return guarded([&] {
        Batch* b = as_batch(batch);
        AGNES_REQUIRE(model, AGNES_ERR_INVALID, "model must not be NULL");
        sage_forward(*b, *model, out, (hipStream_t)hip_stream);
    });
}

agnes_status agnes_sage_forward_noalloc(agnes_batch* batch, const agnes_sage_model* model, float* out,
                                        void* hip_stream) {
    return guarded([&] {
        Batch* b = as_batch(batch);
        AGNES_REQUIRE(model, AGNES_ERR_INVALID, "model must not be NULL");
        sage_forward_noalloc(*b, *model, out, (hipStream_t)hip_stream);
    });
}

agnes_status agnes_batch_tier_stats(const agnes_batch* batch, agnes_tier_stats* out) {
    return guarded([&] {
        Batch* b = as_batch((void*)batch);
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        wait_batch(*b);
        *out = b->tier;
    });
}

agnes_status agnes_store_set_option(agnes_store* store, agnes_option opt, int64_t value) {
    return guarded([&] {
        Store* s = as_store(store);
        if (opt == AGNES_OPT_PROFILE) {
            s->profile = value ? 1 : 0;
        } else if (opt == AGNES_OPT_GATHER_GROUPS) {
            AGNES_REQUIRE(value >= 8 && value <= (1 << 22), AGNES_ERR_INVALID, "gather groups must be in [8, 2^22]");
            s->gather_groups = (int)value;
        } else if (opt == AGNES_OPT_GATHER_UNROLL) {
            AGNES_REQUIRE(value == 0 || value == 4 || value == 8 || value == 16, AGNES_ERR_INVALID,
                          "gather unroll must be 0, 4, 8 or 16");
            s->gather_unroll = (int)value;
        } else if (opt == AGNES_OPT_GATHER_NONTEMPORAL) {
            s->gather_nt = value ? 1 : 0;
        } else if (opt == AGNES_OPT_GATHER_CHUNKS) {
            AGNES_REQUIRE(value >= 1 && value <= 64, AGNES_ERR_INVALID, "gather chunks must be in [1, 64]");
            s->gather_chunks = (int)value;
        } else if (opt == AGNES_OPT_SAMPLING_GRAPH) {
            AGNES_REQUIRE(value >= 0 && value <= 2, AGNES_ERR_INVALID, "sampling graph must be 0, 1 or 2");
            s->sampling_graph = (int)value;
        } else if (opt == AGNES_OPT_JOIN_PATH) {
            AGNES_REQUIRE(value == 0 || value == 1, AGNES_ERR_INVALID, "join path must be 0 or 1");
            s->join_path = (int)value;
        } else if (opt == AGNES_OPT_SAMPLING_GROUPS) {
            AGNES_REQUIRE(value == 0 || (value >= 256 && value <= 4096), AGNES_ERR_INVALID,
                          "sampling groups must be 0 or in [256, 4096]");
            s->sample_groups = (int)value;
        } else if (opt == AGNES_OPT_BUCKET_CAP) {
            AGNES_REQUIRE(value >= 64 && value <= kBucketCap, AGNES_ERR_INVALID, "bucket capacity must be in [64, 2048]");
            s->bucket_cap = (int)value;
        } else {
            throw Error{AGNES_ERR_INVALID, "unknown option"};
        }
    });
}

agnes_status agnes_store_info(const agnes_store* store, int64_t out[8]) {
    return guarded([&] {
        Store* s = as_store((void*)store);
        AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
        out[0] = s->num_nodes;
        out[1] = s->num_edges;
        out[2] = s->nblk;
        out[3] = s->e_blk;
        out[4] = s->nfblk;
        out[5] = s->rpb;
        out[6] = s->row_bytes;
        out[7] = (int64_t)(s->offsets.bytes + s->indices.bytes + s->features.bytes +
                           s->first_node.bytes + s->last_node.bytes + s->pool.bytes + s->tbuf.bytes +
                           s->tch.bytes + s->acc_count.bytes + s->cache_used.bytes);
    });
}

agnes_status agnes_store_object_table(const agnes_store* store, int32_t* first_node,
                                      int32_t* last_node) {
    return guarded([&] {
        Store* s = as_store((void*)store);
        AGNES_REQUIRE(first_node && last_node, AGNES_ERR_INVALID, "outputs must not be NULL");
        AGNES_CHECK_HIP(hipMemcpy(first_node, s->first_node.ptr, (size_t)s->nblk * 4, hipMemcpyDeviceToHost));
        AGNES_CHECK_HIP(hipMemcpy(last_node, s->last_node.ptr, (size_t)s->nblk * 4, hipMemcpyDeviceToHost));
    });
}

agnes_status agnes_philox4x64_10(const uint64_t* counters, const uint64_t* keys, int64_t n, uint64_t* out) {
    return guarded([&] {
        AGNES_REQUIRE(n >= 0 && n <= ((int64_t)1 << 26), AGNES_ERR_INVALID, "n must be in [0, 2^26]");
        if (n == 0) return;
        AGNES_REQUIRE(counters && keys && out, AGNES_ERR_INVALID, "counters, keys and out must not be NULL");
        DevBuf c, k, o;
        c.reserve((size_t)n * 32);
        k.reserve((size_t)n * 16);
        o.reserve((size_t)n * 32);
        AGNES_CHECK_HIP(hipMemcpy(c.ptr, counters, (size_t)n * 32, hipMemcpyHostToDevice));
        AGNES_CHECK_HIP(hipMemcpy(k.ptr, keys, (size_t)n * 16, hipMemcpyHostToDevice));
        philox_words(c.as<uint64_t>(), k.as<uint64_t>(), n, o.as<uint64_t>(), nullptr);
        AGNES_CHECK_HIP(hipMemcpy(out, o.ptr, (size_t)n * 32, hipMemcpyDeviceToHost));
    });
}

agnes_status agnes_set_device_allocator(agnes_device_alloc_fn alloc, agnes_device_free_fn release, void* user) {
    return guarded([&] {
        AGNES_REQUIRE((alloc == nullptr) == (release == nullptr), AGNES_ERR_INVALID,
                      "install both allocator callbacks or neither");
        DeviceAllocator& a = device_allocator();
        a.alloc = alloc;
        a.release = release;
        a.user = alloc ? user : nullptr;
    });
}

void agnes_free(void* handle) {
    if (!handle) return;
    uint32_t magic = *static_cast<uint32_t*>(handle);
    if (magic == kStoreMagic) {
        Store* s = static_cast<Store*>(handle);
        s->magic = 0;
        delete s;
    } else if (magic == kBatchMagic) {
        release_batch(static_cast<Batch*>(handle));
    }
}

const char* agnes_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
