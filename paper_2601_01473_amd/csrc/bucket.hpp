// Node-range buckets of the union and relabel step (bucket.hip): constants,
// the choice of bucket levels (shared by host and device) and host entry
// points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace agnes {

struct Store;
struct Ctl;

constexpr int kBucketCap = 2048;                 // old + new entries of a sorted sub-bucket in LDS
constexpr int kDenseCap = 8192;                  // cells (nodes x minibatches) of a dense sub-bucket
constexpr int kCoarseMax = 1024;                 // coarse buckets of the partition (10-bit digits)
constexpr int kCoarseAvg = 512;                  // entries per coarse bucket aimed at
constexpr int kSubAvg = 1024;                    // entries per sub-bucket aimed at
constexpr int64_t kSubTableMax = (int64_t)16 << 20;   // minibatches x sub-buckets of the count table
constexpr int kMaxBucketLevels = 40;

struct BucketLevels {
    int tc, ts;   // coarse level (the partition's digits) and sub-bucket level
};

// Levels for `load` entries (old list entries plus new records) of a hop with
// H minibatches.  info: [nlev][2] (offset of the level's boundaries, bucket
// count), levels from the finest (0) to the coarsest (one bucket); counts are
// non-increasing.  Coarse: the coarsest level with at least
// min(kCoarseMax, load / kCoarseAvg) buckets, then coarser while above
// kCoarseMax or coarse_cap buckets.  Sub: from the coarse level toward finer
// ones while below load / kSubAvg buckets, as long as the finer level keeps
// H x buckets within kSubTableMax and its buckets within sub_cap.  A smaller
// load never picks a level with more buckets, so bounds computed for an upper
// bound of the load hold for the actual load.
__host__ __device__ inline BucketLevels pick_levels(const int32_t* info, int nlev, int64_t load, int H,
                                                    int64_t coarse_cap, int64_t sub_cap) {
    int64_t want_c = (load + kCoarseAvg - 1) / kCoarseAvg;
    if (want_c > kCoarseMax) want_c = kCoarseMax;
    if (want_c < 1) want_c = 1;
    int tc = nlev - 1;
    while (tc > 0 && info[tc * 2 + 1] < want_c) tc--;
    while (tc < nlev - 1 && (info[tc * 2 + 1] > kCoarseMax || info[tc * 2 + 1] > coarse_cap)) tc++;
    int64_t want_s = (load + kSubAvg - 1) / kSubAvg;
    if (want_s < 1) want_s = 1;
    int ts = tc;
    while (ts > 0 && info[ts * 2 + 1] < want_s && (int64_t)info[(ts - 1) * 2 + 1] * H <= kSubTableMax &&
           info[(ts - 1) * 2 + 1] <= sub_cap)
        ts--;
    BucketLevels lv;
    lv.tc = tc;
    lv.ts = ts;
    return lv;
}

struct BucketBounds {
    int coarse, sub;   // most coarse buckets and sub-buckets a hop of at most `load` entries uses
};

// Builds the store's nested bucket levels from the host index array (in-degree
// weights).
void build_bucket_levels(Store& s, const int32_t* indices, int64_t n, int64_t e);
BucketBounds bucket_bounds(const Store& s, int64_t load, int H);
// Row stride of the per-minibatch count table for those bounds (sub-buckets
// rounded up to a multiple of 256).
inline int bucket_table_stride(const BucketBounds& b) { return (b.sub + 255) / 256 * 256; }

// Records keys[0, *n_dev) reordered by coarse bucket (stable) into kout, with
// their indices into vout; dtot receives the records per coarse bucket and,
// with an old list (ak, *old_dev entries), acoff the old entries before each
// coarse bucket.  n_max / load_max: upper bounds of *n_dev and *n_dev +
// *old_dev; hist: radix_hist_entries(n_max) entries.
void bucket_partition(const uint32_t* keys, uint32_t* kout, uint32_t* vout, const int64_t* n_dev,
                      const int64_t* old_dev, int64_t n_max, int64_t load_max, const Store& s, int H, uint32_t* hist,
                      uint32_t* dtot, const uint64_t* ak, int64_t* acoff, hipStream_t st);

struct BucketJoinArgs {
    const Store* store;
    int H, jbits;
    int write_nodes;            // write new nodes into nodes (another hop follows)
    int64_t capN, rows_cap;
    int cap;                    // entries of a sorted sub-bucket (<= kBucketCap)
    int coarse_max, G;          // grid (coarse buckets) and count-table stride (sub-buckets), host bounds
    const int64_t* n_dev;
    const int64_t* old_dev;
    const uint32_t *rk, *rv, *dtot;
    const int64_t* acoff;
    const uint64_t* ak;
    const int32_t* av;
    const int64_t* req_off;
    const uint32_t* e_off;
    const int32_t* size;
    int64_t *ghist, *gemit, *newcnt;
    int32_t* row_ptr;
    int32_t* nodes;
    uint64_t* ck;
    int32_t* cv;
    int32_t* col;
    Ctl* ctl;
};

// Count pass, scan of the counts, write pass (three launches on st).
void bucket_join(const BucketJoinArgs& j, hipStream_t st);
size_t bucket_lds_bytes(int H);

}  // namespace agnes
