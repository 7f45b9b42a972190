// Node-range buckets of the union and relabel step of every hop (Alg. 1,
// sampling loop: N_out accumulated by union; Sec. 3.4(3), node
// identification).
//
// A hop's sampled edges (u, e) are grouped by node-range bucket in one
// radix-style pass, then each bucket is joined with the pairs (node,
// minibatch) the hyperbatch already holds, which are the entries of the sorted
// list whose node falls in the same range.  A workgroup takes one coarse
// bucket (the partition's digit) and walks its sub-buckets:
//   - a narrow sub-bucket (nodes x minibatches <= kDenseCap cells, e.g. one
//     hub node) is a dense table in LDS indexed by (node, minibatch): its
//     edges are streamed through it, so their number is unbounded;
//   - a wide one is sorted by (node, minibatch) in LDS, up to kBucketCap old
//     and new entries, and merged with its part of the list.
// Both give each new pair (u, j) the local id |S_{j,l-1}| + (new pairs of
// minibatch j in earlier sub-buckets) + (rank among those of this
// sub-bucket), i.e. new nodes ascending by id per minibatch; every edge gets
// the local id of its pair, and the merged list (old and new pairs, ascending
// by (node, minibatch)) is written at the sub-bucket's offset.  A count pass,
// a scan of the counts and a write pass do this in three launches.
//
// Bucket boundaries are fixed per store: nested levels over the node ids,
// each cut where the running weight in-degree(u) + c reaches the level's
// budget, with any node heavier than the budget in a bucket of its own.  The
// levels a hop uses follow from its sizes on the device.  A sorted sub-bucket
// that exceeds its capacity flags the hyperbatch (err bit 3): it keeps its old
// entries only, so the list stays sorted and every size consistent, the later
// hops get no requests, and the host samples the hyperbatch again with the
// radix-sort join (same results).
#include <algorithm>
#include <cstring>
#include <vector>

#include "bucket.hpp"
#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

// ----------------------------------------------------------------- levels (host)

void build_bucket_levels(Store& s, const int32_t* indices, int64_t n, int64_t e) {
    std::vector<uint32_t> indeg((size_t)n, 0u);
    for (int64_t i = 0; i < e; i++) indeg[(size_t)indices[i]]++;
    const double c = std::max(1.0, (double)e / (4.0 * (double)n));
    double W = 0.0;
    for (int64_t u = 0; u < n; u++) W += (double)indeg[(size_t)u] + c;
    int64_t nbf = 1;
    while (nbf * 2 <= 65536 && nbf * 2 * 4 <= n) nbf *= 2;
    // level 0: cut where the running weight reaches the budget; a node heavier
    // than the budget gets a bucket of its own
    std::vector<int32_t> b0{0};
    std::vector<double> w0;
    {
        const double budget = W / (double)nbf;
        double acc = 0.0;
        int64_t start = 0;
        for (int64_t u = 0; u < n; u++) {
            const double wu = (double)indeg[(size_t)u] + c;
            if (wu > budget) {
                if (start < u) {
                    b0.push_back((int32_t)u);
                    w0.push_back(acc);
                }
                b0.push_back((int32_t)(u + 1));
                w0.push_back(wu);
                start = u + 1;
                acc = 0.0;
            } else {
                acc += wu;
                if (acc >= budget) {
                    b0.push_back((int32_t)(u + 1));
                    w0.push_back(acc);
                    start = u + 1;
                    acc = 0.0;
                }
            }
        }
        if (start < n) {
            b0.push_back((int32_t)n);
            w0.push_back(acc);
        }
    }
    // coarser levels: neighbouring buckets merged up to twice the previous
    // budget; a bucket above the new budget stays alone (nested by construction)
    std::vector<std::vector<int32_t>> lev{b0};
    std::vector<double> wcur = w0;
    double budget = W / (double)nbf;
    while (lev.back().size() > 2) {
        budget *= 2.0;
        const std::vector<int32_t>& prev = lev.back();
        std::vector<int32_t> nb{0};
        std::vector<double> nw;
        double acc = 0.0;
        bool open = false;
        for (size_t i = 0; i + 1 < prev.size(); i++) {
            const double wi = wcur[i];
            if (wi > budget) {
                if (open) {
                    nb.push_back(prev[i]);
                    nw.push_back(acc);
                }
                nb.push_back(prev[i + 1]);
                nw.push_back(wi);
                acc = 0.0;
                open = false;
            } else {
                acc += wi;
                open = true;
                if (acc >= budget) {
                    nb.push_back(prev[i + 1]);
                    nw.push_back(acc);
                    acc = 0.0;
                    open = false;
                }
            }
        }
        if (open) {
            nb.push_back((int32_t)n);
            nw.push_back(acc);
        }
        if (nb.size() >= prev.size()) break;   // no merge possible any more
        lev.push_back(std::move(nb));
        wcur = std::move(nw);
    }
    const int nlev = (int)lev.size();
    AGNES_REQUIRE(nlev <= kMaxBucketLevels, AGNES_ERR_INTERNAL, "too many bucket levels");
    std::vector<int32_t> all, info((size_t)nlev * 2);
    for (int t = 0; t < nlev; t++) {
        info[(size_t)t * 2] = (int32_t)all.size();
        info[(size_t)t * 2 + 1] = (int32_t)(lev[t].size() - 1);
        all.insert(all.end(), lev[t].begin(), lev[t].end());
    }
    s.nlev = nlev;
    s.lev_info_host = info;
    s.bnd.reserve(all.size() * 4);
    s.lev_info.reserve(info.size() * 4);
    AGNES_CHECK_HIP(hipMemcpy(s.bnd.ptr, all.data(), all.size() * 4, hipMemcpyHostToDevice));
    AGNES_CHECK_HIP(hipMemcpy(s.lev_info.ptr, info.data(), info.size() * 4, hipMemcpyHostToDevice));
}

// Bucket counts of the levels a hop of `load` old plus new entries may use,
// when its actual load is at most `load`: coarse and sub-bucket maxima.
BucketBounds bucket_bounds(const Store& s, int64_t load, int H) {
    const BucketLevels lv = pick_levels(s.lev_info_host.data(), s.nlev, load, H, INT64_MAX, INT64_MAX);
    BucketBounds b;
    // a smaller load picks coarser (fewer-bucket) levels: the bound is the
    // chosen level's count
    b.coarse = s.lev_info_host[(size_t)lv.tc * 2 + 1];
    b.sub = s.lev_info_host[(size_t)lv.ts * 2 + 1];
    return b;
}

// ----------------------------------------------------------------- partition

// Coarse bucket of node u: the last boundary <= u among bnd[0..nb) (LDS).
__device__ __forceinline__ int coarse_of(const int32_t* bnd, int nb, uint32_t u) {
    int lo = 0, hi = nb;   // bnd[lo] <= u < bnd[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if ((uint32_t)bnd[mid] <= u) lo = mid; else hi = mid;
    }
    return lo;
}

// The coarse level's boundaries into LDS; returns its bucket count.
__device__ __forceinline__ int load_coarse(const int32_t* info, const int32_t* bnd_all, int nlev, int64_t load,
                                           int H, int ccap, int scap, int32_t* lds) {
    const BucketLevels lv = pick_levels(info, nlev, load, H, ccap, scap);
    const int off = info[lv.tc * 2], nb = info[lv.tc * 2 + 1];
    for (int i = threadIdx.x; i <= nb; i += kBlock) lds[i] = bnd_all[off + i];
    __syncthreads();
    return nb;
}

// Per-tile digit histogram, digit = coarse bucket of the key (as k_rs_hist).
template <int ITEMS, int RB>
__global__ __launch_bounds__(kBlock) void k_part_hist(const uint32_t* keys, const int64_t* n_dev, const int64_t* old_dev,
                                                      const int32_t* info, const int32_t* bnd_all, int nlev, int H,
                                                      int ccap, int scap, uint32_t* hist) {
    constexpr int BINS = 1 << RB;
    __shared__ uint32_t h[BINS];
    __shared__ int32_t bnd[BINS + 1];
    const int64_t n = *n_dev;
    const int nb = load_coarse(info, bnd_all, nlev, n + (old_dev ? *old_dev : 0), H, ccap, scap, bnd);
    const int64_t tiles = (n + kBlock * ITEMS - 1) / (kBlock * ITEMS);
    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t t0 = tile * (kBlock * ITEMS);
        __syncthreads();
        for (int d = threadIdx.x; d < BINS; d += kBlock) h[d] = 0;
        uint32_t k[ITEMS];
#pragma unroll
        for (int q = 0; q < ITEMS; q++) {
            const int64_t i = t0 + q * kBlock + threadIdx.x;
            k[q] = i < n ? keys[i] : 0u;
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < ITEMS; q++)
            if (t0 + q * kBlock + threadIdx.x < n) atomicAdd(&h[coarse_of(bnd, nb, k[q])], 1u);
        __syncthreads();
        for (int d = threadIdx.x; d < BINS; d += kBlock) hist[tile * BINS + d] = h[d];
    }
}

// Per coarse bucket d (one workgroup each, dealt to the XCDs in contiguous
// ranges as k_rs_scan): exclusive scan of the tile counts, the digit total,
// and, when there is an old list, the first list entry at or after the
// bucket's first node (one wave's 64-way search).
template <int ITEMS, int RB>
__global__ __launch_bounds__(kBlock) void k_part_scan(uint32_t* hist, const int64_t* n_dev, const int64_t* old_dev,
                                                      const int32_t* info, const int32_t* bnd_all, int nlev, int H,
                                                      int ccap, int scap, uint32_t* dtot, const uint64_t* ak,
                                                      int64_t* acoff) {
    constexpr int BINS = 1 << RB;
    static_assert(BINS % kXcds == 0, "digits split evenly over the XCDs");
    __shared__ uint32_t lds[kWavesPerBlock];
    const int d = (int)(blockIdx.x % kXcds) * (BINS / kXcds) + (int)(blockIdx.x / kXcds);
    const int64_t n = *n_dev;
    const int tiles = (int)((n + (kBlock * ITEMS) - 1) / (kBlock * ITEMS));
    uint32_t carry = 0;
    for (int b0 = 0; b0 < tiles; b0 += kBlock * 4) {
        uint32_t v[4];
        uint32_t local = 0;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const int i = b0 + threadIdx.x * 4 + k;
            v[k] = i < tiles ? hist[(int64_t)i * BINS + d] : 0u;
            local += v[k];
        }
        uint32_t total;
        uint32_t ex = block_exclusive_scan(local, lds, total) + carry;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const int i = b0 + threadIdx.x * 4 + k;
            if (i < tiles) hist[(int64_t)i * BINS + d] = ex;
            ex += v[k];
        }
        carry += total;
    }
    if (threadIdx.x == 0) dtot[d] = carry;
    if (ak && wave_id() == 0) {
        const int64_t na = *old_dev;
        const BucketLevels lv = pick_levels(info, nlev, n + na, H, ccap, scap);
        const int nb = info[lv.tc * 2 + 1];
        if (d <= nb) {
            const uint64_t x = (uint64_t)(uint32_t)bnd_all[info[lv.tc * 2] + d] << 32;
            const int64_t p = wave_partition_point(0, na, [&](int64_t i) { return ak[i] < x; });
            if (lane_id() == 0) acoff[d] = p;
        }
    }
}

// Keys and values reordered by coarse bucket, stable (as k_rs_scatter, with
// the digit looked up in the coarse boundaries); values are the key's index
// (the edge number).
template <int ITEMS, int RB>
__global__ __launch_bounds__(kBlock) void k_part_scatter(const uint32_t* kin, uint32_t* kout, uint32_t* vout,
                                                         const int64_t* n_dev, const int64_t* old_dev,
                                                         const int32_t* info, const int32_t* bnd_all, int nlev, int H,
                                                         int ccap, int scap, const uint32_t* hist,
                                                         const uint32_t* dtot) {
    constexpr int BINS = 1 << RB;
    constexpr int Q = BINS / kBlock;
    static_assert(Q >= 1 && Q * kBlock == BINS, "at least one digit per thread");
    __shared__ uint32_t wcnt[kWavesPerBlock][BINS];
    __shared__ uint32_t lbase[BINS];
    __shared__ uint32_t gbase[BINS];
    __shared__ uint32_t lds[kWavesPerBlock];
    __shared__ uint32_t sk[kBlock * ITEMS];
    __shared__ uint32_t sv[kBlock * ITEMS];
    __shared__ int32_t bnd[BINS + 1];
    const int64_t n = *n_dev;
    const int nb = load_coarse(info, bnd_all, nlev, n + (old_dev ? *old_dev : 0), H, ccap, scap, bnd);
    const int64_t tiles = (n + kBlock * ITEMS - 1) / (kBlock * ITEMS);
    const int64_t per = (tiles + kXcds - 1) / kXcds;
    const int64_t wx = gridDim.x / kXcds;
    const int t = threadIdx.x, w = wave_id(), lane = lane_id();
    for (int64_t local = blockIdx.x / kXcds; local < per; local += wx) {
        const int64_t tile = (int64_t)(blockIdx.x % kXcds) * per + local;
        if (tile >= tiles) break;
        const int64_t t0 = tile * (kBlock * ITEMS);
        __syncthreads();
        for (int x = t; x < kWavesPerBlock * BINS; x += kBlock) (&wcnt[0][0])[x] = 0;
        {
            uint32_t dt[Q], sum = 0;
#pragma unroll
            for (int q = 0; q < Q; q++) {
                dt[q] = dtot[t * Q + q];
                sum += dt[q];
            }
            uint32_t tot;
            uint32_t ex = block_exclusive_scan(sum, lds, tot);
#pragma unroll
            for (int q = 0; q < Q; q++) {
                const int d = t * Q + q;
                gbase[d] = ex + hist[tile * BINS + d];
                ex += dt[q];
            }
        }
        __syncthreads();
        uint32_t key[ITEMS], rnk[ITEMS];
        int dig[ITEMS];
#pragma unroll
        for (int r = 0; r < ITEMS; r++) {
            const int64_t i = t0 + w * (ITEMS * kWave) + r * kWave + lane;
            key[r] = i < n ? kin[i] : 0u;
        }
#pragma unroll
        for (int r = 0; r < ITEMS; r++) {
            const int64_t i = t0 + w * (ITEMS * kWave) + r * kWave + lane;
            const bool valid = i < n;
            const int d = valid ? coarse_of(bnd, nb, key[r]) : -1;
            dig[r] = d;
            uint64_t peers = __ballot(valid);
#pragma unroll
            for (int b = 0; b < RB; b++) {
                const uint64_t m = __ballot((d >> b) & 1);
                peers &= ((d >> b) & 1) ? m : ~m;
            }
            const int rank = __popcll(peers & lanemask_lt());
            const int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane;
            uint32_t old = 0;
            if (valid && rank == 0) {
                old = wcnt[w][d];
                wcnt[w][d] = old + (uint32_t)__popcll(peers);
            }
            old = (uint32_t)__shfl((int)old, leader, kWave);
            rnk[r] = old + rank;
        }
        __syncthreads();
        {
            uint32_t c[Q][kWavesPerBlock], sum = 0;
#pragma unroll
            for (int q = 0; q < Q; q++)
#pragma unroll
                for (int x = 0; x < kWavesPerBlock; x++) {
                    c[q][x] = wcnt[x][t * Q + q];
                    sum += c[q][x];
                }
            uint32_t tot;
            uint32_t ex = block_exclusive_scan(sum, lds, tot);
#pragma unroll
            for (int q = 0; q < Q; q++) {
                const int d = t * Q + q;
                lbase[d] = ex;
#pragma unroll
                for (int x = 0; x < kWavesPerBlock; x++) {
                    wcnt[x][d] = ex;
                    ex += c[q][x];
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < ITEMS; r++) {
            const int64_t i = t0 + w * (ITEMS * kWave) + r * kWave + lane;
            if (i < n) {
                const uint32_t pos = wcnt[w][dig[r]] + rnk[r];
                sk[pos] = key[r];
                sv[pos] = (uint32_t)i;
            }
        }
        __syncthreads();
        const int cnt = (int)((n - t0) < (kBlock * ITEMS) ? (n - t0) : (kBlock * ITEMS));
        for (int i = t; i < cnt; i += kBlock) {
            const uint32_t k = sk[i];
            const int d = coarse_of(bnd, nb, k);
            const uint32_t dst = gbase[d] + (uint32_t)i - lbase[d];
            kout[dst] = k;
            vout[dst] = sv[i];
        }
    }
}

// ----------------------------------------------------------------- bucket join

constexpr int kPerThread = kBucketCap / kBlock;           // sorted entries per thread (8)
constexpr int kRoundsPerWave = kBucketCap / kWavesPerBlock / kWave;
constexpr uint64_t kNoKey = ~0ull;

struct BucketArgs {
    int H, jbits;
    int write_nodes;                // write the new nodes' ids into nodes (another hop follows)
    int64_t capN, rows_cap;
    int cap;                        // entries of a sorted sub-bucket (<= kBucketCap)
    int ccap;                       // coarse buckets the grid covers
    const int32_t* info;            // levels: [nlev][2] (boundary offset, buckets)
    const int32_t* bnd;             // all levels' boundaries
    int nlev;
    const int64_t* n_dev;           // records of the partition (the hop's sampled edges)
    const int64_t* old_dev;         // old list entries (the hop's requests)
    const uint32_t* rk;             // records' nodes, grouped by coarse bucket
    const uint32_t* rv;             // records' edge numbers
    const uint32_t* dtot;           // records per coarse bucket
    const int64_t* acoff;           // old list entries before each coarse bucket
    const uint64_t* ak;             // old list keys (node << 32 | minibatch), sorted
    const int32_t* av;              // old list local ids
    const int64_t* req_off;         // [H+1] requests before minibatch j
    const uint32_t* e_off;          // edge offset of every request
    const int32_t* size;            // nodes of minibatch j before the hop
    int G;                          // row stride of ghist (>= sub-buckets, multiple of kBlock)
    int64_t* ghist;                 // [H][G] new nodes per minibatch and sub-bucket (scanned by k_bkt_scan)
    int64_t* gemit;                 // [G] merged list entries per sub-bucket
    int32_t* row_ptr;               // hop's row pointers (count pass)
    int32_t* nodes;                 // [H][capN] (write pass)
    uint64_t* ck;                   // merged list keys (write pass)
    int32_t* cv;                    // merged list local ids
    int32_t* col;                   // hop's columns, by edge number
    Ctl* ctl;
};

// Dynamic LDS: mb_e[H+1] (int64), per-minibatch cnt[H] (int32), wcnt[4][H]
// (uint16), then the sub-bucket area: the dense table (int32 [kDenseCap]) or
// the sorted entries sk[cap] (uint64), sv[cap], loc[cap], nhx[cap+1] (int32),
// then the sort's per-wave digit counts [4][256] (uint32).
size_t bucket_lds_bytes(int H) {
    size_t b = (size_t)(H + 1) * 8 + (size_t)H * 4 + (size_t)kWavesPerBlock * H * 2;
    b = (b + 15) / 16 * 16;
    const size_t area = std::max<size_t>((size_t)kDenseCap * 4, (size_t)kBucketCap * 20 + 16);
    return b + area + (size_t)kWavesPerBlock * 256 * 4;
}

struct BucketLds {
    int64_t* mb_e;
    int32_t* cnt;
    uint16_t* wcnt;
    int32_t* table;
    uint64_t* sk;
    uint32_t* sv;
    int32_t* loc;
    int32_t* nhx;
    uint32_t (*wd)[256];
};

__device__ __forceinline__ BucketLds carve(int H) {
    extern __shared__ int64_t dyn[];
    BucketLds L;
    char* p = (char*)dyn;
    L.mb_e = (int64_t*)p;
    p += (size_t)(H + 1) * 8;
    L.cnt = (int32_t*)p;
    p += (size_t)H * 4;
    L.wcnt = (uint16_t*)p;
    p += (size_t)kWavesPerBlock * H * 2;
    p = (char*)(((uintptr_t)p + 15) & ~(uintptr_t)15);
    char* area = p;
    L.table = (int32_t*)area;
    L.sk = (uint64_t*)area;
    L.sv = (uint32_t*)(area + (size_t)kBucketCap * 8);
    L.loc = (int32_t*)(area + (size_t)kBucketCap * 12);
    L.nhx = (int32_t*)(area + (size_t)kBucketCap * 16);
    p = area + std::max<size_t>((size_t)kDenseCap * 4, (size_t)kBucketCap * 20 + 16);
    L.wd = (uint32_t(*)[256])p;
    return L;
}

__device__ __forceinline__ int bits_for(uint32_t x) { return x ? 32 - __clz(x) : 0; }

__device__ __forceinline__ int lds_lower_bound64(const uint64_t* a, int lo, int hi, uint64_t key) {
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (a[mid] < key) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// Minibatch (from the edge number) and key (node << 32 | minibatch) of a record.
__device__ __forceinline__ void record_key(const BucketArgs& a, const BucketLds& L, uint32_t u, uint32_t e, int& j,
                                           uint64_t& key) {
    j = upper_segment(L.mb_e, a.H, (int64_t)e);
    key = ((uint64_t)u << 32) | (uint32_t)j;
}

// Stable LSD sort of sk/sv[0, n) by ((node - y0) << jbits | minibatch), 8-bit
// digits ranked by wave ballots (the order of equal digits is kept).
__device__ void lds_sort(uint64_t* sk, uint32_t* sv, int n, uint32_t y0, int jbits, int nbits, uint32_t (*wd)[256],
                         int32_t* scan_lds) {
    const int w = wave_id(), lane = lane_id(), t = threadIdx.x;
    const uint64_t jmask = ((uint64_t)1 << jbits) - 1;
    for (int shift = 0; shift < nbits; shift += 8) {
        for (int x = t; x < kWavesPerBlock * 256; x += kBlock) (&wd[0][0])[x] = 0;
        uint64_t key[kPerThread];
        uint32_t val[kPerThread], rnk[kPerThread];
        int dig[kPerThread];
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kPerThread; r++) {
            const int i = w * (kPerThread * kWave) + r * kWave + lane;
            const bool valid = i < n;
            key[r] = valid ? sk[i] : 0;
            val[r] = valid ? sv[i] : 0;
            const uint64_t sortkey = ((uint64_t)((uint32_t)(key[r] >> 32) - y0) << jbits) | (key[r] & jmask);
            const int d = valid ? (int)((sortkey >> shift) & 255) : -1;
            dig[r] = d;
            uint64_t peers = __ballot(valid);
#pragma unroll
            for (int b = 0; b < 8; b++) {
                const uint64_t m = __ballot((d >> b) & 1);
                peers &= ((d >> b) & 1) ? m : ~m;
            }
            const int rank = __popcll(peers & lanemask_lt());
            const int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane;
            uint32_t old = 0;
            if (valid && rank == 0) {
                old = wd[w][d];
                wd[w][d] = old + (uint32_t)__popcll(peers);
            }
            old = (uint32_t)__shfl((int)old, leader, kWave);
            rnk[r] = old + rank;
        }
        __syncthreads();
        {
            // thread t owns digit t: wave prefixes and the digit's start
            uint32_t c[kWavesPerBlock], sum = 0;
#pragma unroll
            for (int x = 0; x < kWavesPerBlock; x++) {
                c[x] = wd[x][t];
                sum += c[x];
            }
            int32_t tot;
            int32_t ex = block_exclusive_scan((int32_t)sum, scan_lds, tot);
#pragma unroll
            for (int x = 0; x < kWavesPerBlock; x++) {
                wd[x][t] = (uint32_t)ex;
                ex += (int32_t)c[x];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kPerThread; r++) {
            if (dig[r] >= 0) {
                const uint32_t pos = wd[w][dig[r]] + rnk[r];
                sk[pos] = key[r];
                sv[pos] = val[r];
            }
        }
        __syncthreads();
    }
}

// First old list entry in [lo, hi) with key >= x (one wave; all its lanes).
__device__ __forceinline__ int64_t old_lower_bound(const uint64_t* ak, int64_t lo, int64_t hi, uint64_t x) {
    return wave_partition_point(lo, hi, [&](int64_t i) { return ak[i] < x; });
}

template <bool WRITE>
__device__ void sub_bucket(const BucketArgs& a, const BucketLds& L, int sidx, uint32_t y0, uint32_t y1, int64_t r0,
                           int64_t r1, int64_t a0, int64_t a1, bool dense, int32_t* scan_lds, int64_t* s64,
                           int32_t* s32) {
    const int H = a.H, t = threadIdx.x, w = wave_id(), lane = lane_id();
    const int64_t nA = a1 - a0;
    const uint32_t width = y1 - y0;
    // merged output offset of the sub-bucket (write pass)
    const int64_t m0 = WRITE ? a.gemit[sidx] : 0;
    if (dense) {
        // -------- dense: cell (u - y0) * H + j; -1 absent, -2 new, else a local id
        const int cells = (int)width * H;
        for (int c = t; c < cells; c += kBlock) L.table[c] = -1;
        __syncthreads();
        for (int64_t i = a0 + t; i < a1; i += kBlock) {
            const uint64_t K = a.ak[i];
            L.table[(int)((uint32_t)(K >> 32) - y0) * H + (int)(uint32_t)K] = a.av[i];
        }
        __syncthreads();
        for (int64_t p = r0 + t; p < r1; p += kBlock) {
            const uint32_t u = a.rk[p];
            if (u < y0 || u >= y1) continue;
            int j;
            uint64_t K;
            record_key(a, L, u, a.rv[p], j, K);
            const int c = (int)(u - y0) * H + j;
            if (L.table[c] == -1) L.table[c] = -2;
        }
        __syncthreads();
        if (!WRITE) {
            // new cells per minibatch, present cells in all
            int present = 0;
            for (int c = t; c < cells; c += kBlock) {
                const int32_t v = L.table[c];
                if (v != -1) present++;
                if (v == -2) atomicAdd(&L.cnt[c % H], 1);
            }
            int32_t tot;
            (void)block_exclusive_scan(present, scan_lds, tot);
            if (t == 0) a.gemit[sidx] = tot;
            __syncthreads();
            for (int j = t; j < H; j += kBlock) {
                a.ghist[(int64_t)j * a.G + sidx] = L.cnt[j];
                L.cnt[j] = 0;
            }
            __syncthreads();
            return;
        }
        // local ids of the new cells: per minibatch, ascending node
        for (int j = t; j < H; j += kBlock) {
            int32_t next = a.size[j] + (int32_t)a.ghist[(int64_t)j * a.G + sidx];
            for (int r = 0; r < (int)width; r++) {
                const int c = r * H + j;
                if (L.table[c] == -2) {
                    if (next >= a.capN) atomicOr((unsigned long long*)&a.ctl->err, 4ull);
                    L.table[c] = next;
                    if (a.write_nodes && next < a.capN) a.nodes[(int64_t)j * a.capN + next] = (int32_t)(y0 + r);
                    next++;
                }
            }
        }
        __syncthreads();
        // merged list: present cells in (node, minibatch) order; each thread
        // owns a contiguous run of cells
        const int per = (cells + kBlock - 1) / kBlock;
        const int c0 = std::min(cells, t * per), c1 = std::min(cells, c0 + per);
        int mine = 0;
        for (int c = c0; c < c1; c++) mine += L.table[c] != -1 ? 1 : 0;
        int32_t tot;
        int32_t pos = block_exclusive_scan(mine, scan_lds, tot);
        for (int c = c0; c < c1; c++) {
            const int32_t v = L.table[c];
            if (v == -1) continue;
            const int64_t q = m0 + pos++;
            if (q < a.rows_cap) {
                a.ck[q] = ((uint64_t)(y0 + (uint32_t)(c / H)) << 32) | (uint32_t)(c % H);
                a.cv[q] = v;
            } else {
                atomicOr((unsigned long long*)&a.ctl->err, 4ull);
            }
        }
        // every edge's column
        for (int64_t p = r0 + t; p < r1; p += kBlock) {
            const uint32_t u = a.rk[p];
            if (u < y0 || u >= y1) continue;
            const uint32_t e = a.rv[p];
            int j;
            uint64_t K;
            record_key(a, L, u, e, j, K);
            a.col[e] = L.table[(int)(u - y0) * H + j];
        }
        __syncthreads();
        return;
    }
    // -------- sorted: old entries in sk[0, nA), this sub-bucket's records after them
    uint64_t* skA = L.sk;
    uint32_t* svA = L.sv;
    const bool a_fits = nA <= a.cap;
    if (a_fits)
        for (int64_t i = t; i < nA; i += kBlock) {
            skA[i] = a.ak[a0 + i];
            svA[i] = (uint32_t)a.av[a0 + i];
        }
    if (t == 0) s32[0] = 0;
    __syncthreads();
    const int capB = a_fits ? a.cap - (int)nA : 0;
    for (int64_t base = r0; base < r1; base += kBlock) {
        const int64_t p = base + t;
        uint32_t u = 0, e = 0;
        bool in = false;
        if (p < r1) {
            u = a.rk[p];
            in = u >= y0 && u < y1;
            if (in) e = a.rv[p];
        }
        const uint64_t m = __ballot(in);
        if (lane == 0) s32[1 + w] = __popcll(m);
        __syncthreads();
        int before = s32[0];
        for (int x = 0; x < w; x++) before += s32[1 + x];
        const int pos = before + __popcll(m & lanemask_lt());
        if (in && pos < capB) {
            int j;
            uint64_t K;
            record_key(a, L, u, e, j, K);
            skA[nA + pos] = K;
            svA[nA + pos] = e;
        }
        __syncthreads();
        if (t == 0) s32[0] += s32[1] + s32[2] + s32[3] + s32[4];
        __syncthreads();
    }
    const int nB = s32[0];
    if (!a_fits || nB > capB) {
        // over capacity: the hyperbatch is sampled again on the other path;
        // until then the sub-bucket keeps its old entries only (no new
        // nodes), so the list stays sorted and every size consistent
        if (t == 0) atomicOr((unsigned long long*)&a.ctl->err, 8ull);
        if (!WRITE) {
            if (t == 0) a.gemit[sidx] = nA;
            for (int j = t; j < H; j += kBlock) a.ghist[(int64_t)j * a.G + sidx] = 0;
        } else {
            for (int64_t i = t; i < nA; i += kBlock)
                if (m0 + i < a.rows_cap) {
                    a.ck[m0 + i] = a.ak[a0 + i];
                    a.cv[m0 + i] = a.av[a0 + i];
                }
        }
        __syncthreads();
        return;
    }
    uint64_t* skB = skA + nA;
    uint32_t* svB = svA + nA;
    lds_sort(skB, svB, nB, y0, a.jbits, bits_for(width - 1) + a.jbits, L.wd, scan_lds);
    if (!WRITE) {
        int nh = 0;
        for (int i = t; i < nB; i += kBlock) {
            const uint64_t K = skB[i];
            if (i > 0 && skB[i - 1] == K) continue;
            const int idx = lds_lower_bound64(skA, 0, (int)nA, K);
            if (idx < nA && skA[idx] == K) continue;
            atomicAdd(&L.cnt[(uint32_t)K], 1);
            nh++;
        }
        int32_t tot;
        (void)block_exclusive_scan(nh, scan_lds, tot);
        if (t == 0) a.gemit[sidx] = nA + tot;
        __syncthreads();
        for (int j = t; j < H; j += kBlock) {
            a.ghist[(int64_t)j * a.G + sidx] = L.cnt[j];
            L.cnt[j] = 0;
        }
        __syncthreads();
        return;
    }
    // write pass: wave w takes entries [w R 64, (w + 1) R 64) in rounds of 64.
    // A head (first entry of a key) whose key the old entries hold takes that
    // local id; a new head takes cursor[j] + (new heads of minibatch j before
    // it), ranked by ballots within a round, rounds in order and waves by
    // their counts.
    for (int j = t; j < H; j += kBlock) {
        L.cnt[j] = a.size[j] + (int32_t)a.ghist[(int64_t)j * a.G + sidx];
        for (int x = 0; x < kWavesPerBlock; x++) L.wcnt[x * H + j] = 0;
    }
    __syncthreads();
    const uint64_t lane_le = lanemask_lt() | (1ull << lane);
    uint64_t key[kRoundsPerWave];
    int32_t nhw[kRoundsPerWave], jrk[kRoundsPerWave], anc[kRoundsPerWave], idx[kRoundsPerWave], floc[kRoundsPerWave];
    uint32_t kind = 0;
    int nh_run = 0, anc_run = -1;
#pragma unroll
    for (int r = 0; r < kRoundsPerWave; r++) {
        const int i = w * (kRoundsPerWave * kWave) + r * kWave + lane;
        const bool valid = i < nB;
        const uint64_t K = valid ? skB[i] : 0;
        bool head = false, found = false;
        int id = 0;
        int32_t fl = 0;
        if (valid) {
            head = i == 0 || skB[i - 1] != K;
            if (head) {
                id = lds_lower_bound64(skA, 0, (int)nA, K);
                if (id < nA && skA[id] == K) {
                    found = true;
                    fl = (int32_t)svA[id];
                }
            }
        }
        const bool nh = head && !found;
        const uint64_t nhm = __ballot(nh);
        nhw[r] = nh_run + __popcll(nhm & lanemask_lt());
        nh_run += __popcll(nhm);
        const int j = (int)(uint32_t)K;
        uint64_t peers = nhm;
        for (int bit = 0; bit < a.jbits; bit++) {
            const uint64_t m = __ballot((j >> bit) & 1);
            peers &= ((j >> bit) & 1) ? m : ~m;
        }
        const int rank = __popcll(peers & lanemask_lt());
        const int leader = nh ? (__ffsll((unsigned long long)peers) - 1) : lane;
        int old = 0;
        if (nh && rank == 0) {
            old = L.wcnt[w * H + j];
            L.wcnt[w * H + j] = (uint16_t)(old + __popcll(peers));
        }
        old = __shfl(old, leader, kWave);
        jrk[r] = old + rank;
        const uint64_t hm = __ballot(head);
        const uint64_t le = hm & lane_le;
        const int base = w * (kRoundsPerWave * kWave) + r * kWave;
        anc[r] = le ? base + 63 - __clzll(le) : anc_run;
        if (hm) anc_run = base + 63 - __clzll(hm);
        key[r] = K;
        idx[r] = id;
        floc[r] = fl;
        kind |= ((head ? 1u : 0u) | (nh ? 2u : 0u)) << (2 * r);
    }
    int32_t* wnh = s32 + 8;
    int32_t* wanc = s32 + 16;
    if (lane == 0) {
        wnh[w] = nh_run;
        wanc[w] = anc_run;
    }
    __syncthreads();
    int nh_base = 0, nh_total = 0, anc_carry = -1;
#pragma unroll
    for (int x = 0; x < kWavesPerBlock; x++) {
        if (x < w) {
            nh_base += wnh[x];
            anc_carry = std::max(anc_carry, wanc[x]);
        }
        nh_total += wnh[x];
    }
#pragma unroll
    for (int r = 0; r < kRoundsPerWave; r++) {
        const int i = w * (kRoundsPerWave * kWave) + r * kWave + lane;
        if (i >= nB) continue;
        L.nhx[i] = nh_base + nhw[r];
        if (anc[r] < 0) anc[r] = anc_carry;
        if ((kind >> (2 * r)) & 1u) {
            int32_t lc = floc[r];
            if ((kind >> (2 * r)) & 2u) {
                const int j = (int)(uint32_t)key[r];
                int rank = jrk[r];
                for (int x = 0; x < w; x++) rank += L.wcnt[x * H + j];
                lc = L.cnt[j] + rank;
                const int64_t pos = m0 + idx[r] + nh_base + nhw[r];
                if (lc >= a.capN || pos >= a.rows_cap) {
                    atomicOr((unsigned long long*)&a.ctl->err, 4ull);
                } else {
                    if (a.write_nodes) a.nodes[(int64_t)j * a.capN + lc] = (int32_t)(key[r] >> 32);
                    a.ck[pos] = key[r];
                    a.cv[pos] = lc;
                }
            }
            L.loc[i] = lc;
        }
    }
    if (t == 0) L.nhx[nB] = nh_total;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRoundsPerWave; r++) {
        const int i = w * (kRoundsPerWave * kWave) + r * kWave + lane;
        if (i < nB) a.col[svB[i]] = L.loc[anc[r]];
    }
    for (int ia = t; ia < nA; ia += kBlock) {
        const uint64_t K = skA[ia];
        const int lb = lds_lower_bound64(skB, 0, nB, K);
        const int64_t pos = m0 + ia + L.nhx[lb];
        if (pos < a.rows_cap) {
            a.ck[pos] = K;
            a.cv[pos] = (int32_t)svA[ia];
        }
    }
    __syncthreads();
}

// One workgroup per coarse bucket (blockIdx < the hop's coarse count): its
// records [r0, r1) and old entries [A0, A1), taken whole when they fit one
// sorted sub-bucket or the whole bucket is narrow enough for a dense table,
// else sub-bucket by sub-bucket of the finer level.  The results of a bucket
// taken whole go to its first sub-bucket's slot (the others count zero).
// The count pass also writes the hop's row pointers.
template <bool WRITE>
__global__ __launch_bounds__(kBlock) void k_bkt(BucketArgs a) {
    const BucketLds L = carve(a.H);
    __shared__ int32_t scan_lds[kWavesPerBlock];
    __shared__ int64_t s64[4];
    __shared__ int32_t s32[24];
    const int H = a.H, t = threadIdx.x;
    const int64_t n = *a.n_dev;
    const int64_t na = a.old_dev ? *a.old_dev : 0;
    const BucketLevels lv = pick_levels(a.info, a.nlev, n + na, H, a.ccap, a.G);
    const int nbc = a.info[lv.tc * 2 + 1], offc = a.info[lv.tc * 2];
    const int nbs = a.info[lv.ts * 2 + 1], offs = a.info[lv.ts * 2];
    for (int i = t; i <= H; i += kBlock) L.mb_e[i] = (int64_t)a.e_off[a.req_off[i]];
    if (!WRITE) {
        // row pointers in request order: row r of minibatch j starts at its
        // edge offset minus the minibatch's first edge
        const int64_t R = na;
        __syncthreads();
        for (int64_t q = (int64_t)blockIdx.x * kBlock + t; q < R; q += (int64_t)gridDim.x * kBlock) {
            const int j = upper_segment(a.req_off, H, q);
            a.row_ptr[q + j] = (int32_t)((int64_t)a.e_off[q] - L.mb_e[j]);
            if (q + 1 == a.req_off[j + 1]) a.row_ptr[q + j + 1] = (int32_t)((int64_t)a.e_off[q + 1] - L.mb_e[j]);
        }
    }
    for (int j = t; j < H; j += kBlock) L.cnt[j] = 0;
    __syncthreads();
    const int c = blockIdx.x;
    if (c >= nbc) return;
    // the bucket's records: digit totals before it
    {
        int64_t before = 0;
        for (int d = t; d < c; d += kBlock) before += a.dtot[d];
        int64_t tot;
        int64_t ex = block_exclusive_scan(before, s64, tot);
        (void)ex;
        if (t == 0) s64[0] = tot;
        __syncthreads();
    }
    const int64_t r0 = s64[0], r1 = r0 + a.dtot[c];
    const int64_t A0 = a.acoff[c], A1 = c + 1 < nbc ? a.acoff[c + 1] : na;
    const uint32_t x0 = (uint32_t)a.bnd[offc + c], x1 = (uint32_t)a.bnd[offc + c + 1];
    // sub-buckets of the finer level inside [x0, x1): nested, so exact
    int s0 = 0, s1 = 0;
    {
        const int32_t* bs = a.bnd + offs;
        int lo = 0, hi = nbs;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if ((uint32_t)bs[mid] < x0) lo = mid + 1; else hi = mid;
        }
        s0 = lo;
        hi = nbs;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if ((uint32_t)bs[mid] < x1) lo = mid + 1; else hi = mid;
        }
        s1 = lo;
    }
    const bool whole_dense = (int64_t)(x1 - x0) * H <= kDenseCap;
    const bool whole = whole_dense || (r1 - r0) + (A1 - A0) <= a.cap || s1 - s0 <= 1;
    if (whole) {
        if (!WRITE)
            for (int s = s0 + 1 + t; s < s1; s += kBlock) {
                a.gemit[s] = 0;
                for (int j = 0; j < H; j++) a.ghist[(int64_t)j * a.G + s] = 0;
            }
        sub_bucket<WRITE>(a, L, s0, x0, x1, r0, r1, A0, A1, whole_dense, scan_lds, s64, s32);
        return;
    }
    const int32_t* bs = a.bnd + offs;
    int64_t ap = A0;
    for (int s = s0; s < s1; s++) {
        const uint32_t y0 = (uint32_t)bs[s], y1 = (uint32_t)bs[s + 1];
        int64_t ae = A1;
        if (s + 1 < s1) {
            if (wave_id() == 0) {
                const int64_t p = old_lower_bound(a.ak, ap, A1, (uint64_t)y1 << 32);
                if (lane_id() == 0) s64[1] = p;
            }
            __syncthreads();
            ae = s64[1];
            __syncthreads();
        }
        const bool dense = (int64_t)(y1 - y0) * H <= kDenseCap;
        sub_bucket<WRITE>(a, L, s, y0, y1, r0, r1, ap, ae, dense, scan_lds, s64, s32);
        ap = ae;
    }
}

// Per minibatch j (workgroup j < H): exclusive scan of its new-node counts
// over the sub-buckets and its total; workgroup H: the same for the merged
// entries, and the hop's new-node total (merged entries minus the old list).
__global__ __launch_bounds__(kBlock) void k_bkt_scan(int H, int rows, int ccap, int G, const int32_t* info, int nlev,
                                                     const int64_t* n_dev, const int64_t* old_dev, int64_t* ghist,
                                                     int64_t* gemit, int64_t* newcnt, Ctl* ctl) {
    __shared__ int64_t lds[kWavesPerBlock];
    const int x = blockIdx.x;
    const int64_t na = old_dev ? *old_dev : 0;
    const BucketLevels lv = pick_levels(info, nlev, *n_dev + na, H, ccap, G);
    const int nbs = info[lv.ts * 2 + 1];
    int64_t* row = x < rows ? ghist + (int64_t)x * G : gemit;
    int64_t carry = 0;
    for (int b0 = 0; b0 < nbs; b0 += kBlock * 4) {
        int64_t v[4], local = 0;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const int i = b0 + threadIdx.x * 4 + k;
            v[k] = i < nbs ? row[i] : 0;
            local += v[k];
        }
        int64_t total;
        int64_t ex = block_exclusive_scan(local, lds, total) + carry;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const int i = b0 + threadIdx.x * 4 + k;
            if (i < nbs) row[i] = ex;
            ex += v[k];
        }
        carry += total;
    }
    if (threadIdx.x == 0) {
        if (x < rows) newcnt[x] = carry;
        else if (ctl) ctl->n_new = carry - na;
    }
}

// ----------------------------------------------------------------- host launches

template <int ITEMS, int RB>
static void partition_rb(const uint32_t* keys, uint32_t* kout, uint32_t* vout, const int64_t* n_dev,
                         const int64_t* old_dev, const Store& s, int H, int ccap, int scap, int tiles, uint32_t* hist,
                         uint32_t* dtot, const uint64_t* ak, int64_t* acoff, hipStream_t st) {
    const int grid = std::min(2048, (tiles + kXcds - 1) / kXcds * kXcds);
    const int32_t* info = s.lev_info.as<int32_t>();
    const int32_t* bnd = s.bnd.as<int32_t>();
    AGNES_LAUNCH((k_part_hist<ITEMS, RB>), dim3(grid), dim3(kBlock), 0, st, keys, n_dev, old_dev, info, bnd,
                 s.nlev, H, ccap, scap, hist);
    AGNES_LAUNCH((k_part_scan<ITEMS, RB>), dim3(1 << RB), dim3(kBlock), 0, st, hist, n_dev, old_dev, info, bnd,
                 s.nlev, H, ccap, scap, dtot, ak, acoff);
    AGNES_LAUNCH((k_part_scatter<ITEMS, RB>), dim3(grid), dim3(kBlock), 0, st, keys, kout, vout, n_dev, old_dev,
                 info, bnd, s.nlev, H, ccap, scap, hist, dtot);
}

void bucket_partition(const uint32_t* keys, uint32_t* kout, uint32_t* vout, const int64_t* n_dev,
                      const int64_t* old_dev, int64_t n_max, int64_t load_max, const Store& s, int H, uint32_t* hist,
                      uint32_t* dtot, const uint64_t* ak, int64_t* acoff, hipStream_t st) {
    const BucketBounds bb = bucket_bounds(s, load_max, H);
    const int ccap = bb.coarse, scap = bucket_table_stride(bb);
    const bool wide = bb.coarse > 256;   // 10-bit digits for more than 256 coarse buckets
    const int tiles = (int)radix_tiles(n_max);
    if (radix_items(n_max) == 8) {
        if (wide) partition_rb<8, 10>(keys, kout, vout, n_dev, old_dev, s, H, ccap, scap, tiles, hist, dtot, ak, acoff, st);
        else partition_rb<8, 8>(keys, kout, vout, n_dev, old_dev, s, H, ccap, scap, tiles, hist, dtot, ak, acoff, st);
    } else {
        if (wide) partition_rb<16, 10>(keys, kout, vout, n_dev, old_dev, s, H, ccap, scap, tiles, hist, dtot, ak, acoff, st);
        else partition_rb<16, 8>(keys, kout, vout, n_dev, old_dev, s, H, ccap, scap, tiles, hist, dtot, ak, acoff, st);
    }
}

void bucket_join(const BucketJoinArgs& j, hipStream_t st) {
    BucketArgs a{};
    a.H = j.H;
    a.jbits = j.jbits;
    a.write_nodes = j.write_nodes;
    a.capN = j.capN;
    a.rows_cap = j.rows_cap;
    a.cap = j.cap;
    a.ccap = j.coarse_max;
    a.info = j.store->lev_info.as<int32_t>();
    a.bnd = j.store->bnd.as<int32_t>();
    a.nlev = j.store->nlev;
    a.n_dev = j.n_dev;
    a.old_dev = j.old_dev;
    a.rk = j.rk;
    a.rv = j.rv;
    a.dtot = j.dtot;
    a.acoff = j.acoff;
    a.ak = j.ak;
    a.av = j.av;
    a.req_off = j.req_off;
    a.e_off = j.e_off;
    a.size = j.size;
    a.G = j.G;
    a.ghist = j.ghist;
    a.gemit = j.gemit;
    a.row_ptr = j.row_ptr;
    a.nodes = j.nodes;
    a.ck = j.ck;
    a.cv = j.cv;
    a.col = j.col;
    a.ctl = j.ctl;
    const size_t lds = bucket_lds_bytes(j.H);
    const int grid = std::max(1, j.coarse_max);
    AGNES_LAUNCH(k_bkt<false>, dim3(grid), dim3(kBlock), lds, st, a);
    AGNES_LAUNCH(k_bkt_scan, dim3(j.H + 1), dim3(kBlock), 0, st, j.H, j.H, j.coarse_max, j.G, a.info, a.nlev,
                 j.n_dev, j.old_dev, j.ghist, j.gemit, j.newcnt, j.ctl);
    AGNES_LAUNCH(k_bkt<true>, dim3(grid), dim3(kBlock), lds, st, a);
}

}  // namespace agnes
