// Block store: the CSR topology and the feature matrix as fixed-size pages in
// HBM, and the object index table (Sec. 3.2(1) storage layer, Sec. 3.2(2)).
//
// Topology block b holds edges [b * E_blk, (b + 1) * E_blk) of the index array,
// E_blk = block_bytes / 4.  The object of node v is its adjacency list
// [off[v], off[v+1]); its home block is the one holding its first edge, so
// objects are laid out in ascending node order and a long list continues into
// the following blocks.  Feature block c holds rows [c * rpb, (c + 1) * rpb),
// rpb = floor(block_bytes / row_bytes).  Both arrays are padded to whole blocks.
#include <cstdlib>
#include <cstring>
#include <memory>
#include <vector>

#include "bucket.hpp"
#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

// first_node[b] / last_node[b]: the first and last node whose home block is b
// (home is nondecreasing in v, so each block's objects form one id range).
template <typename OffT>
__global__ __launch_bounds__(kBlock) void k_object_table(const OffT* off, int64_t n, int e_blk_log2,
                                                         int64_t nblk, int32_t* first_node,
                                                         int32_t* last_node) {
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < n; v += (int64_t)gridDim.x * kBlock) {
        auto home = [&](int64_t x) {
            int64_t b = (int64_t)off[x] >> e_blk_log2;
            return b < nblk ? b : nblk - 1;
        };
        int64_t b = home(v);
        if (v == 0 || home(v - 1) != b) first_node[b] = (int32_t)v;
        if (v == n - 1 || home(v + 1) != b) last_node[b] = (int32_t)v;
    }
}

static int dtype_size(agnes_dtype d) {
    switch (d) {
        case AGNES_FLOAT32: return 4;
        case AGNES_FLOAT16: return 2;
        case AGNES_BFLOAT16: return 2;
        default: return 0;
    }
}

template <typename OffT>
static int64_t validate_offsets(const OffT* off, int64_t n, int64_t e) {
    AGNES_REQUIRE(off[0] == 0, AGNES_ERR_INVALID, "offsets[0] must be 0");
    int64_t maxdeg = 0;
    for (int64_t v = 0; v < n; v++) {
        int64_t d = (int64_t)off[v + 1] - (int64_t)off[v];
        AGNES_REQUIRE(d >= 0, AGNES_ERR_INVALID, "offsets must be nondecreasing");
        if (d > maxdeg) maxdeg = d;
    }
    AGNES_REQUIRE((int64_t)off[n] == e, AGNES_ERR_INVALID, "offsets[num_nodes] must equal num_edges");
    return maxdeg;
}

Store* build_store(const agnes_csr* csr, const agnes_features* feat, uint64_t block_bytes,
                   int64_t pool_blocks, int64_t cache_rows, int64_t cache_threshold, hipStream_t st) {
    Range range("agnes_build_blocks");
    AGNES_REQUIRE(pool_blocks >= 0, AGNES_ERR_INVALID, "pool_blocks must not be negative");
    AGNES_REQUIRE(cache_rows >= 0, AGNES_ERR_INVALID, "cache_rows must not be negative");
    AGNES_REQUIRE(cache_threshold >= 1, AGNES_ERR_INVALID, "the cache threshold must be >= 1");
    AGNES_REQUIRE(csr && feat, AGNES_ERR_INVALID, "csr and features must not be NULL");
    const int64_t n = csr->num_nodes, e = csr->num_edges;
    AGNES_REQUIRE(n >= 1 && n < 0x7FFFFFFFll, AGNES_ERR_INVALID, "num_nodes must be in [1, 2^31-1)");
    AGNES_REQUIRE(e >= 0, AGNES_ERR_INVALID, "num_edges must be >= 0");
    AGNES_REQUIRE(csr->offsets, AGNES_ERR_INVALID, "offsets must not be NULL");
    AGNES_REQUIRE(csr->indices || e == 0, AGNES_ERR_INVALID, "indices must not be NULL");
    AGNES_REQUIRE(csr->offsets_dtype == AGNES_INT32 || csr->offsets_dtype == AGNES_INT64,
                  AGNES_ERR_INVALID, "offsets dtype must be AGNES_INT32 or AGNES_INT64");
    AGNES_REQUIRE(feat->data, AGNES_ERR_INVALID, "feature data must not be NULL");
    const int ds = dtype_size(feat->dtype);
    AGNES_REQUIRE(ds > 0, AGNES_ERR_INVALID, "feature dtype must be FLOAT32, FLOAT16 or BFLOAT16");
    AGNES_REQUIRE(feat->dim >= 1 && feat->dim <= (1 << 24), AGNES_ERR_INVALID, "feature dim out of range");
    const int64_t row_bytes = feat->dim * ds;
    AGNES_REQUIRE(row_bytes % 4 == 0, AGNES_ERR_INVALID, "row_bytes must be a multiple of 4");
    AGNES_REQUIRE(block_bytes >= 16 && block_bytes <= (1u << 24) && (block_bytes & (block_bytes - 1)) == 0,
                  AGNES_ERR_INVALID, "block_bytes must be a power of two in [16, 2^24]");
    AGNES_REQUIRE((int64_t)block_bytes >= row_bytes, AGNES_ERR_INVALID, "block_bytes must be >= row_bytes");

    const bool o64 = csr->offsets_dtype == AGNES_INT64;
    if (!o64) AGNES_REQUIRE(e < 0x7FFFFFFFll, AGNES_ERR_INVALID, "int32 offsets need num_edges < 2^31");
    int64_t maxdeg = o64 ? validate_offsets((const int64_t*)csr->offsets, n, e)
                         : validate_offsets((const int32_t*)csr->offsets, n, e);
    AGNES_REQUIRE(maxdeg < 0x7FFFFFFFll, AGNES_ERR_INVALID, "a node has >= 2^31 edges");
    for (int64_t i = 0; i < e; i++) {
        int32_t u = csr->indices[i];
        if (u < 0 || u >= n) throw Error{AGNES_ERR_INVALID, "indices[" + std::to_string(i) + "] out of range"};
    }

    std::unique_ptr<Store> s(new Store());
    AGNES_CHECK_HIP(hipGetDevice(&s->device));
    AGNES_CHECK_HIP(hipDeviceGetAttribute(&s->max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, s->device));
    s->num_nodes = n;
    s->num_edges = e;
    // int64 offsets of a graph with fewer than 2^31 edges are kept on the
    // device as int32: the same values in half the bytes, so more of them
    // share a cache line in the samplers' random reads.  AGNES_WIDE_OFFSETS=1
    // keeps them as given (so that the int64 kernels can be tested on small
    // graphs).
    const char* wide = std::getenv("AGNES_WIDE_OFFSETS");
    const bool narrow = o64 && e < 0x7FFFFFFFll && !(wide && wide[0] == '1');
    s->offsets64 = (o64 && !narrow) ? 1 : 0;
    s->block_bytes = (int64_t)block_bytes;
    s->e_blk = (int64_t)block_bytes / 4;
    s->e_blk_log2 = 0;
    while (((int64_t)1 << s->e_blk_log2) < s->e_blk) s->e_blk_log2++;
    s->nblk = e > 0 ? (e + s->e_blk - 1) / s->e_blk : 1;
    s->row_bytes = row_bytes;
    s->feat_dtype = feat->dtype;
    s->rpb = (int64_t)block_bytes / row_bytes;
    s->nfblk = (n + s->rpb - 1) / s->rpb;
    s->max_degree = maxdeg;
    s->node_bits = 1;
    while (((int64_t)1 << s->node_bits) < n) s->node_bits++;

    const size_t obytes = (size_t)(n + 1) * (s->offsets64 ? 8 : 4);
    const size_t ibytes = (size_t)(s->nblk * s->e_blk) * 4;
    const size_t fbytes = (size_t)(s->nfblk * s->rpb) * (size_t)row_bytes;
    const size_t fdata = (size_t)n * (size_t)row_bytes;
    s->offsets.reserve(obytes);
    s->indices.reserve(ibytes);
    s->first_node.reserve((size_t)s->nblk * 4);
    s->last_node.reserve((size_t)s->nblk * 4);
    if (narrow) {
        // a synchronous copy from pageable memory: o32 outlives it
        const int64_t* src = (const int64_t*)csr->offsets;
        std::vector<int32_t> o32((size_t)n + 1);
        for (int64_t i = 0; i <= n; i++) o32[i] = (int32_t)src[i];
        AGNES_CHECK_HIP(hipStreamSynchronize(st));
        AGNES_CHECK_HIP(hipMemcpy(s->offsets.ptr, o32.data(), obytes, hipMemcpyHostToDevice));
    } else {
        AGNES_CHECK_HIP(hipMemcpyAsync(s->offsets.ptr, csr->offsets, obytes, hipMemcpyHostToDevice, st));
    }
    if (e > 0)
        AGNES_CHECK_HIP(hipMemcpyAsync(s->indices.ptr, csr->indices, (size_t)e * 4, hipMemcpyHostToDevice, st));
    if (ibytes > (size_t)e * 4)
        AGNES_CHECK_HIP(hipMemsetAsync((char*)s->indices.ptr + (size_t)e * 4, 0, ibytes - (size_t)e * 4, st));
    if (pool_blocks > 0) {
        // the storage tier: the padded feature matrix in pinned host memory,
        // read by the GPU through its mapped address; HBM holds only the pool
        s->tiered = 1;
        s->pool_blocks = pool_blocks;
        AGNES_CHECK_HIP(hipHostMalloc(&s->host_feat, fbytes, hipHostMallocMapped));
        memcpy(s->host_feat, feat->data, fdata);
        if (fbytes > fdata) memset((char*)s->host_feat + fdata, 0, fbytes - fdata);
        AGNES_CHECK_HIP(hipHostGetDevicePointer(&s->host_feat_dev, s->host_feat, 0));
        s->pool_rows = pool_blocks * s->rpb;
        s->cache_rows = cache_rows;
        s->cache_threshold = cache_threshold;
        s->pool.reserve((size_t)(s->pool_rows + cache_rows) * (size_t)row_bytes);
        s->tbuf.reserve((size_t)s->nfblk * 4);
        fill_u32(s->tbuf.ptr, 0xFFFFFFFFu, s->nfblk, st);
        if (cache_rows > 0) {
            s->tch.reserve((size_t)n * 4);
            s->acc_count.reserve((size_t)n * 4);
            s->cache_used.reserve(8);
            fill_u32(s->tch.ptr, 0xFFFFFFFFu, n, st);
            fill_u32(s->acc_count.ptr, 0u, n, st);
            fill_u32(s->cache_used.ptr, 0u, 2, st);
        }
        s->slot_block.assign((size_t)pool_blocks, -1);
        s->slot_stamp.assign((size_t)pool_blocks, -1);
        s->block_slot.assign((size_t)s->nfblk, -1);
        AGNES_CHECK_HIP(hipEventCreateWithFlags(&s->pool_free, hipEventDisableTiming));
        AGNES_CHECK_HIP(hipEventRecord(s->pool_free, st));
    } else {
        s->features.reserve(fbytes);
        AGNES_CHECK_HIP(hipMemcpyAsync(s->features.ptr, feat->data, fdata, hipMemcpyHostToDevice, st));
        if (fbytes > fdata)
            AGNES_CHECK_HIP(hipMemsetAsync((char*)s->features.ptr + fdata, 0, fbytes - fdata, st));
    }
    fill_u32(s->first_node.ptr, 0xFFFFFFFFu, s->nblk, st);
    fill_u32(s->last_node.ptr, 0xFFFFFFFFu, s->nblk, st);
    if (s->offsets64)
        AGNES_LAUNCH(k_object_table<int64_t>, dim3(grid_for(n, 4096)), dim3(kBlock), 0, st,
                           s->offsets.as<int64_t>(), n, s->e_blk_log2, s->nblk,
                           s->first_node.as<int32_t>(), s->last_node.as<int32_t>());
    else
        AGNES_LAUNCH(k_object_table<int32_t>, dim3(grid_for(n, 4096)), dim3(kBlock), 0, st,
                           s->offsets.as<int32_t>(), n, s->e_blk_log2, s->nblk,
                           s->first_node.as<int32_t>(), s->last_node.as<int32_t>());
    AGNES_CHECK_HIP(hipGetLastError());
    AGNES_CHECK_HIP(hipStreamSynchronize(st));
    build_bucket_levels(*s, csr->indices, n, e);
    return s.release();
}

}  // namespace agnes
