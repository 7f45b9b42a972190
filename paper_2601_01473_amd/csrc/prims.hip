// Device-wide primitives: fill, exclusive scan and stable LSD radix sort of
// (key, value) pairs.  Element counts are read from device memory, so a launch
// sequence never waits for the host to learn a size; the host only supplies an
// upper bound for the buffers.
#include <algorithm>

#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

// ----------------------------------------------------------------- fill

__global__ void k_fill_u32(uint32_t* p, uint32_t value, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock)
        p[i] = value;
}

void fill_u32(void* p, uint32_t value, int64_t n, hipStream_t st) {
    if (n <= 0) return;
    AGNES_LAUNCH(k_fill_u32, dim3(grid_for(n, 2048)), dim3(kBlock), 0, st, (uint32_t*)p, value, n);
    AGNES_CHECK_HIP(hipGetLastError());
}

// ----------------------------------------------------------------- Philox words

// The sampler's generator on given counters and keys ([n][4] and [n][2]), for
// checking it against the published definition.
__global__ void k_philox_words(const uint64_t* c, const uint64_t* k, int64_t n, uint64_t* out) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) {
        const Words4 w = philox4x64_10(c[4 * i], c[4 * i + 1], c[4 * i + 2], c[4 * i + 3], k[2 * i], k[2 * i + 1]);
        for (int q = 0; q < 4; q++) out[4 * i + q] = w.w[q];
    }
}

void philox_words(const uint64_t* c, const uint64_t* k, int64_t n, uint64_t* out, hipStream_t st) {
    if (n <= 0) return;
    AGNES_LAUNCH(k_philox_words, dim3(grid_for(n, 1024)), dim3(kBlock), 0, st, c, k, n, out);
    AGNES_CHECK_HIP(hipGetLastError());
}

// ----------------------------------------------------------------- scan

int64_t scan_partials_needed() { return kScanGroups + 1; }

template <typename T>
__global__ void k_scan_reduce(const T* in, const int64_t* n_dev, int G, int64_t* partials,
                              int64_t* nonzero) {
    __shared__ int64_t lds[kWavesPerBlock];
    __shared__ int64_t ldz[kWavesPerBlock];
    int64_t lo, hi;
    scan_range(*n_dev, G, blockIdx.x, lo, hi);
    int64_t s = 0, z = 0;
    for (int64_t i = lo + threadIdx.x; i < hi; i += kBlock) {
        T x = in[i];
        s += (int64_t)x;
        z += (x != 0) ? 1 : 0;
    }
    s = wave_inclusive_scan(s);
    z = wave_inclusive_scan(z);
    if (lane_id() == kWave - 1) {
        lds[wave_id()] = s;
        ldz[wave_id()] = z;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0, tz = 0;
        for (int w = 0; w < kWavesPerBlock; w++) {
            t += lds[w];
            tz += ldz[w];
        }
        partials[blockIdx.x] = t;
        if (nonzero && tz) atomicAdd((unsigned long long*)nonzero, (unsigned long long)tz);
    }
}

// Each block adds the partial sums of the blocks before it itself (G <=
// kScanGroups = 4 * kBlock: four per thread), so no separate launch scans
// them; block 0 also writes the total after the last element and to
// total_dev.
template <typename T, typename OutT>
__global__ void k_scan_final(const T* in, OutT* out, const int64_t* n_dev, int G,
                             const int64_t* partials, int64_t* total_dev) {
    __shared__ int64_t lds[kWavesPerBlock];
    const int64_t n = *n_dev;
    int64_t lo, hi;
    scan_range(n, G, blockIdx.x, lo, hi);
    int64_t before = 0, all = 0;
    for (int k = 0; k < 4; k++) {
        const int i = threadIdx.x * 4 + k;
        const int64_t v = (i < G) ? partials[i] : 0;
        all += v;
        if (i < (int)blockIdx.x) before += v;
    }
    int64_t carry, total;
    (void)block_exclusive_scan(before, lds, carry);
    __syncthreads();                                  // lds is reused
    (void)block_exclusive_scan(all, lds, total);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        out[n] = (OutT)total;
        if (total_dev) *total_dev = total;
    }
    for (int64_t base = lo; base < hi; base += kScanTile) {
        int64_t v[kScanItems];
        int64_t local = 0;
#pragma unroll
        for (int k = 0; k < kScanItems; k++) {
            int64_t i = base + (int64_t)threadIdx.x * kScanItems + k;
            v[k] = (i < hi) ? (int64_t)in[i] : 0;
            local += v[k];
        }
        int64_t total;
        int64_t ex = block_exclusive_scan(local, lds, total);
        ex += carry;
#pragma unroll
        for (int k = 0; k < kScanItems; k++) {
            int64_t i = base + (int64_t)threadIdx.x * kScanItems + k;
            if (i < hi) out[i] = (OutT)ex;
            ex += v[k];
        }
        carry += total;
    }
}

int scan_groups(int64_t n_max) {
    const int64_t g = (n_max + kScanTile - 1) / kScanTile;
    return (int)(g < 1 ? 1 : (g > kScanGroups ? kScanGroups : g));
}

void scan_counts_final(const int32_t* in, uint32_t* out, const int64_t* n_dev, int64_t n_max, int64_t* total_dev,
                       const int64_t* partials, hipStream_t st) {
    const int G = scan_groups(n_max);
    AGNES_LAUNCH((k_scan_final<int32_t, uint32_t>), dim3(G), dim3(kBlock), 0, st, in, out, n_dev, G, partials,
                 total_dev);
}

template <typename T>
static void scan_impl(const T* in, int64_t* out, const int64_t* n_dev, int64_t n_max,
                      int64_t* total_dev, int64_t* partials, int64_t* nonzero, hipStream_t st) {
    const int G = scan_groups(n_max);
    AGNES_LAUNCH(k_scan_reduce<T>, dim3(G), dim3(kBlock), 0, st, in, n_dev, G, partials, nonzero);
    AGNES_LAUNCH((k_scan_final<T, int64_t>), dim3(G), dim3(kBlock), 0, st, in, out, n_dev, G, partials, total_dev);
    AGNES_CHECK_HIP(hipGetLastError());
}

void scan_counts(const int32_t* in, int64_t* out, const int64_t* n_dev, int64_t n_max,
                 int64_t* total_dev, int64_t* partials, hipStream_t st, int64_t* nonzero) {
    scan_impl<int32_t>(in, out, n_dev, n_max, total_dev, partials, nonzero, st);
}

// ----------------------------------------------------------------- radix sort

// LSD radix sort of 32-bit keys with 32-bit values, tiles of 256 x ITEMS keys
// (2048 for sorts of at most 2M keys, where more and shorter workgroups hide
// latency better; 4096 above, and 8192 above 8M keys with 8-bit digits, for
// longer runs per digit).  Digits are RB = 8,
// 9 or 10 bits, the fewest passes that cover the key bits with digits of at
// most 10 bits: 20-bit keys take two passes of 10, 26-bit keys three of 9,
// 23-bit keys three of 8.  Per pass: (1) digit histogram of every tile, stored
// tile-major (each tile writes its counts contiguously), (2) per digit, an
// exclusive scan over the tiles (the table is small and stays in L2), (3) each
// tile ranks its keys stably, reorders them by digit in LDS and writes every
// digit's run contiguously.
constexpr int64_t kSmallSort = 1 << 21;
static int sort_items(int64_t n_max) { return n_max <= kSmallSort ? 8 : 16; }
int radix_items(int64_t n_max) { return sort_items(n_max); }
// Sorts of more than kLargeSort keys with 8-bit digits take tiles of 8192
// keys: a digit's run is then 32 keys on average, a whole 128-byte line of
// keys, where 4096-key tiles leave half lines behind.  (With 9- or 10-bit
// digits the runs stay shorter than a line, and the larger tiles only cost
// occupancy: 2 workgroups per CU.)  Tile counts, and so the histogram, stay
// below the 4096-key sizing above.
constexpr int64_t kLargeSort = (int64_t)1 << 23;
constexpr int kMaxRadixBits = 10;

// Tiles rounded up to a multiple of the XCD count (the scatter's grid).
static int64_t scatter_grid_tiles(int64_t tiles) { return (tiles + kXcds - 1) / kXcds * kXcds; }

int64_t radix_tiles(int64_t n_max) {
    const int64_t tile = (int64_t)kBlock * sort_items(n_max);
    return (n_max + tile - 1) / tile + 1;
}
// Histogram entries for any sort of at most n_max keys: tiles are shorter up
// to kSmallSort keys, so a smaller sort can need more tiles than a larger one.
int64_t radix_hist_entries(int64_t n_max) {
    const int64_t tiles = std::max(radix_tiles(std::min(n_max, kSmallSort)), radix_tiles(n_max));
    return ((int64_t)1 << kMaxRadixBits) * scatter_grid_tiles(tiles);
}
int64_t radix_dtot_entries() { return (int64_t)1 << kMaxRadixBits; }

template <int ITEMS, int RB>
__global__ __launch_bounds__(kBlock) void k_rs_hist(const uint32_t* keys, const int64_t* n_dev, int shift,
                                                    uint32_t* hist) {
    constexpr int BINS = 1 << RB;
    __shared__ uint32_t h[BINS];
    const int64_t n = *n_dev;
    const int64_t tiles = (n + kBlock * ITEMS - 1) / (kBlock * ITEMS);
    // a tile's keys are loaded while the previous tile is counted and written
    uint32_t k[ITEMS];
    auto load = [&](int64_t tile) {
        const int64_t t0 = tile * (kBlock * ITEMS);
#pragma unroll
        for (int q = 0; q < ITEMS; q++) {
            const int64_t i = t0 + q * kBlock + threadIdx.x;
            k[q] = i < n ? keys[i] : 0u;
        }
    };
    if (blockIdx.x < tiles) load(blockIdx.x);
    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t t0 = tile * (kBlock * ITEMS);
        __syncthreads();                        // the previous tile's counts are written out
        for (int d = threadIdx.x; d < BINS; d += kBlock) h[d] = 0;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < ITEMS; q++)
            if (t0 + q * kBlock + threadIdx.x < n) atomicAdd(&h[(k[q] >> shift) & (BINS - 1)], 1u);
        if (tile + gridDim.x < tiles) load(tile + gridDim.x);
        __syncthreads();
        for (int d = threadIdx.x; d < BINS; d += kBlock) hist[tile * BINS + d] = h[d];
    }
}

// One workgroup per digit: exclusive scan over the tiles that hold keys of
// column d of the tile-major table (in place), digit total.  Neighbouring
// digits share cache lines of the table, and workgroups are dealt to the 8
// XCDs (each with its own L2) in turn, so XCD x is given the contiguous digits
// [x BINS / 8, (x + 1) BINS / 8): a line is then read into one L2, not eight.
template <int ITEMS, int RB>
__global__ __launch_bounds__(kBlock) void k_rs_scan(uint32_t* hist, const int64_t* n_dev, uint32_t* dtot) {
    constexpr int BINS = 1 << RB;
    static_assert(BINS % kXcds == 0, "digits split evenly over the XCDs");
    __shared__ uint32_t lds[kWavesPerBlock];
    const int d = (int)(blockIdx.x % kXcds) * (BINS / kXcds) + (int)(blockIdx.x / kXcds);
    const int tiles = (int)((*n_dev + (kBlock * ITEMS) - 1) / (kBlock * ITEMS));
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
}

// Wave w ranks a quarter of the tile's keys in ITEMS rounds of 64; ranks
// inside a round follow lane order (ballot match), rounds follow each other, and
// waves follow each other, so equal digits keep their input order.  Thread t
// owns digits [t Q, (t + 1) Q), Q = BINS / 256, in the per-digit scans.
// Consecutive tiles write consecutive pieces of every digit's run, so their
// partial cache lines are shared; workgroups are dealt to the XCDs in turn, so
// XCD x takes the contiguous tiles [x per, (x + 1) per), per = ceil(tiles / 8),
// and those lines fill up in one L2.  The grid is a multiple of 8 workgroups;
// the workgroups of one XCD take its tiles in turn.
template <int ITEMS, int RB>
__global__ __launch_bounds__(kBlock) void k_rs_scatter(const uint32_t* kin, const uint32_t* vin,
                                                       uint32_t* kout, uint32_t* vout, const int64_t* n_dev,
                                                       int shift, const uint32_t* hist, const uint32_t* dtot) {
    constexpr int BINS = 1 << RB;
    constexpr int Q = BINS / kBlock;
    static_assert(Q >= 1 && Q * kBlock == BINS, "at least one digit per thread");
    __shared__ uint32_t wcnt[kWavesPerBlock][BINS];
    __shared__ uint32_t lbase[BINS];
    __shared__ uint32_t gbase[BINS];
    __shared__ uint32_t lds[kWavesPerBlock];
    __shared__ uint32_t sk[kBlock * ITEMS];
    __shared__ uint32_t sv[kBlock * ITEMS];
    const int64_t n = *n_dev;
    const int64_t tiles = (n + kBlock * ITEMS - 1) / (kBlock * ITEMS);
    const int64_t per = (tiles + kXcds - 1) / kXcds;
    const int64_t wx = gridDim.x / kXcds;          // workgroups of one XCD
    const int t = threadIdx.x, w = wave_id(), lane = lane_id();
    // a tile's keys and values are loaded while the previous tile is written
    uint32_t key[ITEMS], val[ITEMS], rnk[ITEMS];
    auto load = [&](int64_t tile) {
        const int64_t t0 = tile * (kBlock * ITEMS);
#pragma unroll
        for (int r = 0; r < ITEMS; r++) {
            int64_t i = t0 + w * (ITEMS * kWave) + r * kWave + lane;
            key[r] = i < n ? kin[i] : 0u;
            val[r] = i < n ? (vin ? vin[i] : (uint32_t)i) : 0u;
        }
    };
    {
        const int64_t first = (int64_t)(blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
        if (blockIdx.x / kXcds < per && first < tiles) load(first);
    }
    for (int64_t local = blockIdx.x / kXcds; local < per; local += wx) {
    const int64_t tile = (int64_t)(blockIdx.x % kXcds) * per + local;
    if (tile >= tiles) break;
    const int64_t t0 = tile * (kBlock * ITEMS);
    __syncthreads();                               // the previous tile's LDS is consumed
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
#pragma unroll
    for (int r = 0; r < ITEMS; r++) {
        int64_t i = t0 + w * (ITEMS * kWave) + r * kWave + lane;
        bool valid = i < n;
        int d = valid ? (int)((key[r] >> shift) & (BINS - 1)) : -1;
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < RB; b++) {
            uint64_t m = __ballot((d >> b) & 1);
            peers &= ((d >> b) & 1) ? m : ~m;
        }
        int rank = __popcll(peers & lanemask_lt());
        int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane;
        uint32_t old = 0;
        if (valid && rank == 0) {
            old = wcnt[w][d];
            wcnt[w][d] = old + (uint32_t)__popcll(peers);
        }
        old = (uint32_t)__shfl((int)old, leader, kWave);
        rnk[r] = old + rank;
    }
    __syncthreads();
    // per digit: wave prefixes and the tile's digit offsets
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
        if (t0 + w * (ITEMS * kWave) + r * kWave + lane < n) {
            uint32_t pos = wcnt[w][(key[r] >> shift) & (BINS - 1)] + rnk[r];
            sk[pos] = key[r];
            sv[pos] = val[r];
        }
    }
    {
        const int64_t next = (int64_t)(blockIdx.x % kXcds) * per + local + wx;
        if (local + wx < per && next < tiles) load(next);
    }
    __syncthreads();
    const int cnt = (int)((n - t0) < (kBlock * ITEMS) ? (n - t0) : (kBlock * ITEMS));
    for (int i = t; i < cnt; i += kBlock) {
        uint32_t k = sk[i];
        int d = (int)((k >> shift) & (BINS - 1));
        uint32_t dst = gbase[d] + (uint32_t)i - lbase[d];
        kout[dst] = k;
        vout[dst] = sv[i];
    }
    }
}

// Workgroups of the histogram and scatter kernels for at most `tiles` tiles:
// at most kRadixGroups, which loop over the tiles.  The grid is sized from the
// hop's upper bound while the keys actually sorted are often far fewer, and
// beside a long kernel of another stream every workgroup, even one that finds
// no tile, waits for a slot: a capped grid keeps such kernels short.  A
// multiple of 8 (the scatter splits its workgroups evenly over the XCDs).
constexpr int kRadixGroups = 2048;
static int radix_grid(int tiles, int cap) {
    const int c = std::max(kXcds, std::min(kRadixGroups, cap) / kXcds * kXcds);
    return std::min(c, (tiles + kXcds - 1) / kXcds * kXcds);
}

template <int ITEMS, int RB>
static void radix_passes(uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                         const int64_t* n_dev, int tiles, int passes, uint32_t* hist, uint32_t* dtot,
                         hipStream_t st, bool vals_iota, int cap) {
    uint32_t *ka = keys, *kb = keys_tmp;
    uint32_t *va = vals, *vb = vals_tmp;
    for (int p = 0; p < passes; p++) {
        int shift = p * RB;
        const uint32_t* vin = (p == 0 && vals_iota) ? nullptr : va;
        AGNES_LAUNCH((k_rs_hist<ITEMS, RB>), dim3(radix_grid(tiles, cap)), dim3(kBlock), 0, st, ka, n_dev, shift,
                           hist);
        AGNES_LAUNCH((k_rs_scan<ITEMS, RB>), dim3(1 << RB), dim3(kBlock), 0, st, hist, n_dev, dtot);
        AGNES_LAUNCH((k_rs_scatter<ITEMS, RB>), dim3(radix_grid(tiles, cap)), dim3(kBlock), 0, st, ka, vin, kb,
                           vb, n_dev, shift, hist, dtot);
        uint32_t* tk = ka; ka = kb; kb = tk;
        uint32_t* tv = va; va = vb; vb = tv;
    }
}

template <int ITEMS>
static void radix_passes_rb(int rb, uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                            const int64_t* n_dev, int tiles, int passes, uint32_t* hist, uint32_t* dtot,
                            hipStream_t st, bool vals_iota, int cap) {
    if (rb == 8)
        radix_passes<ITEMS, 8>(keys, vals, keys_tmp, vals_tmp, n_dev, tiles, passes, hist, dtot, st, vals_iota, cap);
    else if (rb == 9)
        radix_passes<ITEMS, 9>(keys, vals, keys_tmp, vals_tmp, n_dev, tiles, passes, hist, dtot, st, vals_iota, cap);
    else
        radix_passes<ITEMS, 10>(keys, vals, keys_tmp, vals_tmp, n_dev, tiles, passes, hist, dtot, st, vals_iota, cap);
}

int radix_sort_pairs32(uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                       const int64_t* n_dev, int64_t n_max, int bits, uint32_t* hist,
                       uint32_t* dtot, hipStream_t st, bool vals_iota, int max_groups) {
    if (bits < 1) bits = 1;
    // the fewest passes with digits of at most 10 bits, then the narrowest
    // digit (at least 8 bits) that covers the key in that many passes
    const int passes = (bits + kMaxRadixBits - 1) / kMaxRadixBits;
    const int rb = std::max(8, (bits + passes - 1) / passes);
    const int tiles = (int)radix_tiles(n_max);
    if (sort_items(n_max) == 8)
        radix_passes_rb<8>(rb, keys, vals, keys_tmp, vals_tmp, n_dev, tiles, passes, hist, dtot, st, vals_iota,
                           max_groups);
    else if (n_max > kLargeSort && rb == 8)
        radix_passes<32, 8>(keys, vals, keys_tmp, vals_tmp, n_dev, (int)((n_max + 8191) / 8192 + 1), passes, hist,
                            dtot, st, vals_iota, max_groups);
    else
        radix_passes_rb<16>(rb, keys, vals, keys_tmp, vals_tmp, n_dev, tiles, passes, hist, dtot, st, vals_iota,
                            max_groups);
    AGNES_CHECK_HIP(hipGetLastError());
    return passes & 1;   // 1: the sorted pairs are in keys_tmp / vals_tmp
}

}  // namespace agnes
