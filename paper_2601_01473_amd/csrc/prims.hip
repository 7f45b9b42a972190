// Device-wide primitives: fill, exclusive scan and stable LSD radix sort of
// (key, value) pairs.  Element counts are read from device memory, so a launch
// sequence never waits for the host to learn a size; the host only supplies an
// upper bound for the buffers.
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
    hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(n, 2048)), dim3(kBlock), 0, st, (uint32_t*)p, value, n);
    AGNES_CHECK_HIP(hipGetLastError());
}

// ----------------------------------------------------------------- scan

constexpr int kScanGroups = 1024;   // partial sums per scan
constexpr int kScanItems = 4;       // consecutive elements per thread per tile
constexpr int kScanTile = kBlock * kScanItems;

int64_t scan_partials_needed() { return kScanGroups + 1; }

__device__ __forceinline__ void scan_range(int64_t n, int G, int g, int64_t& lo, int64_t& hi) {
    int64_t chunk = (n + G - 1) / G;
    chunk = (chunk + kScanTile - 1) / kScanTile * kScanTile;
    lo = (int64_t)g * chunk;
    if (lo > n) lo = n;
    hi = lo + chunk;
    if (hi > n) hi = n;
}

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

__global__ void k_scan_top(int64_t* partials, int G, const int64_t* n_dev, int64_t* out,
                           int64_t* total_dev) {
    __shared__ int64_t lds[kWavesPerBlock];
    // G <= kScanGroups = 4 * kBlock: four consecutive partials per thread
    int64_t v[4];
    int64_t local = 0;
    for (int k = 0; k < 4; k++) {
        int i = threadIdx.x * 4 + k;
        v[k] = (i < G) ? partials[i] : 0;
        local += v[k];
    }
    int64_t total;
    int64_t ex = block_exclusive_scan(local, lds, total);
    for (int k = 0; k < 4; k++) {
        int i = threadIdx.x * 4 + k;
        if (i < G) partials[i] = ex;
        ex += v[k];
    }
    if (threadIdx.x == 0) {
        out[*n_dev] = total;
        if (total_dev) *total_dev = total;
    }
}

template <typename T>
__global__ void k_scan_final(const T* in, int64_t* out, const int64_t* n_dev, int G,
                             const int64_t* partials) {
    __shared__ int64_t lds[kWavesPerBlock];
    int64_t lo, hi;
    scan_range(*n_dev, G, blockIdx.x, lo, hi);
    int64_t carry = partials[blockIdx.x];
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
            if (i < hi) out[i] = ex;
            ex += v[k];
        }
        carry += total;
    }
}

template <typename T>
static void scan_impl(const T* in, int64_t* out, const int64_t* n_dev, int64_t n_max,
                      int64_t* total_dev, int64_t* partials, int64_t* nonzero, hipStream_t st) {
    int64_t g = (n_max + kScanTile - 1) / kScanTile;
    int G = (int)(g < 1 ? 1 : (g > kScanGroups ? kScanGroups : g));
    hipLaunchKernelGGL(k_scan_reduce<T>, dim3(G), dim3(kBlock), 0, st, in, n_dev, G, partials, nonzero);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, st, partials, G, n_dev, out, total_dev);
    hipLaunchKernelGGL(k_scan_final<T>, dim3(G), dim3(kBlock), 0, st, in, out, n_dev, G, partials);
    AGNES_CHECK_HIP(hipGetLastError());
}

void scan_counts(const int32_t* in, int64_t* out, const int64_t* n_dev, int64_t n_max,
                 int64_t* total_dev, int64_t* partials, hipStream_t st, int64_t* nonzero) {
    scan_impl<int32_t>(in, out, n_dev, n_max, total_dev, partials, nonzero, st);
}

void scan_counts64(const int64_t* in, int64_t* out, const int64_t* n_dev, int64_t n_max,
                   int64_t* total_dev, int64_t* partials, hipStream_t st, int64_t* nonzero) {
    scan_impl<int64_t>(in, out, n_dev, n_max, total_dev, partials, nonzero, st);
}

// ----------------------------------------------------------------- radix sort

constexpr int kSortGroups = 512;     // workgroups per pass; each owns a contiguous range
constexpr int kMaxDigitBits = 11;
constexpr int kMaxBins = 1 << kMaxDigitBits;
int64_t radix_hist_entries() { return (int64_t)kMaxBins * kSortGroups; }
int64_t radix_dtot_entries() { return kMaxBins; }

__device__ __forceinline__ void sort_range(int64_t n, int g, int64_t& lo, int64_t& hi) {
    int64_t chunk = (n + kSortGroups - 1) / kSortGroups;
    lo = (int64_t)g * chunk;
    if (lo > n) lo = n;
    hi = lo + chunk;
    if (hi > n) hi = n;
}

// Digit histogram of each workgroup's range: hist[d * kSortGroups + g].
__global__ __launch_bounds__(kBlock) void k_rs_hist(const uint64_t* keys, const int64_t* n_dev,
                                                    int shift, int dbits, int64_t* hist) {
    __shared__ uint32_t h[kMaxBins];
    const int nb = 1 << dbits;
    for (int d = threadIdx.x; d < nb; d += kBlock) h[d] = 0;
    __syncthreads();
    int64_t lo, hi;
    sort_range(*n_dev, blockIdx.x, lo, hi);
    for (int64_t i = lo + threadIdx.x; i < hi; i += kBlock)
        atomicAdd(&h[(keys[i] >> shift) & (uint64_t)(nb - 1)], 1u);
    __syncthreads();
    for (int d = threadIdx.x; d < nb; d += kBlock) hist[(int64_t)d * kSortGroups + blockIdx.x] = h[d];
}

// Per digit d (one workgroup each): exclusive scan over the workgroups, digit total.
__global__ __launch_bounds__(kBlock) void k_rs_scan(int64_t* hist, int64_t* dtot) {
    __shared__ int64_t lds[kWavesPerBlock];
    int64_t* row = hist + (int64_t)blockIdx.x * kSortGroups;
    constexpr int per = kSortGroups / kBlock;
    int64_t v[per];
    int64_t local = 0;
#pragma unroll
    for (int k = 0; k < per; k++) {
        v[k] = row[threadIdx.x * per + k];
        local += v[k];
    }
    int64_t total;
    int64_t ex = block_exclusive_scan(local, lds, total);
#pragma unroll
    for (int k = 0; k < per; k++) {
        row[threadIdx.x * per + k] = ex;
        ex += v[k];
    }
    if (threadIdx.x == 0) dtot[blockIdx.x] = total;
}

// Stable scatter in rounds of 256 consecutive keys.  Inside a wave, keys with the
// same digit are matched with ballots (rank = lane order); the waves then take
// their digit ranges from the running cursors one after the other (wave order),
// so equal digits keep their input order.
__global__ __launch_bounds__(kBlock) void k_rs_scatter(const uint64_t* kin, const uint32_t* vin,
                                                       uint64_t* kout, uint32_t* vout,
                                                       const int64_t* n_dev, int shift, int dbits,
                                                       const int64_t* hist, const int64_t* dtot) {
    __shared__ int64_t cursor[kMaxBins];
    __shared__ int64_t lds[kWavesPerBlock];
    const int nb = 1 << dbits;
    const int t = threadIdx.x;
    const int g = blockIdx.x;
    // digit bases: exclusive scan of the digit totals, plus this group's offset
    int64_t carry = 0;
    for (int d0 = 0; d0 < nb; d0 += kBlock) {
        int d = d0 + t;
        int64_t v = (d < nb) ? dtot[d] : 0;
        int64_t total;
        int64_t ex = block_exclusive_scan(v, lds, total);
        if (d < nb) cursor[d] = carry + ex + hist[(int64_t)d * kSortGroups + g];
        carry += total;
    }
    int64_t lo, hi;
    sort_range(*n_dev, g, lo, hi);
    __syncthreads();
    for (int64_t base = lo; base < hi; base += kBlock) {
        int64_t i = base + t;
        bool valid = i < hi;
        uint64_t key = valid ? kin[i] : 0;
        uint32_t val = valid ? vin[i] : 0;
        int d = (int)((key >> shift) & (uint64_t)(nb - 1));
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < dbits; b++) {
            uint64_t m = __ballot((d >> b) & 1);
            peers &= ((d >> b) & 1) ? m : ~m;
        }
        int rank = __popcll(peers & lanemask_lt());
        int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane_id();
        int64_t dbase = 0;
        for (int w = 0; w < kWavesPerBlock; w++) {
            if (wave_id() == w) {
                if (valid && rank == 0) {
                    dbase = cursor[d];
                    cursor[d] = dbase + __popcll(peers);
                }
                dbase = (int64_t)shfl64((uint64_t)dbase, leader);
            }
            __syncthreads();
        }
        if (valid) {
            int64_t dst = dbase + rank;
            kout[dst] = key;
            vout[dst] = val;
        }
    }
}

int radix_sort_pairs(uint64_t* keys, uint32_t* vals, uint64_t* keys_tmp, uint32_t* vals_tmp,
                     const int64_t* n_dev, int64_t n_max, int bits, int64_t* hist,
                     int64_t* dtot, hipStream_t st) {
    (void)n_max;
    if (bits < 1) bits = 1;
    int passes = (bits + kMaxDigitBits - 1) / kMaxDigitBits;
    int dbits = (bits + passes - 1) / passes;
    uint64_t *ka = keys, *kb = keys_tmp;
    uint32_t *va = vals, *vb = vals_tmp;
    for (int p = 0; p < passes; p++) {
        int shift = p * dbits;
        hipLaunchKernelGGL(k_rs_hist, dim3(kSortGroups), dim3(kBlock), 0, st, ka, n_dev, shift, dbits, hist);
        hipLaunchKernelGGL(k_rs_scan, dim3(1 << dbits), dim3(kBlock), 0, st, hist, dtot);
        hipLaunchKernelGGL(k_rs_scatter, dim3(kSortGroups), dim3(kBlock), 0, st, ka, va, kb, vb,
                           n_dev, shift, dbits, hist, dtot);
        uint64_t* tk = ka; ka = kb; kb = tk;
        uint32_t* tv = va; va = vb; vb = tv;
    }
    AGNES_CHECK_HIP(hipGetLastError());
    return passes & 1;   // 1: the sorted pairs are in keys_tmp / vals_tmp
}

}  // namespace agnes
