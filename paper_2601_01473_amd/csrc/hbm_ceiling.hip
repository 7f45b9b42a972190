// HBM ceiling probe: what plain streaming kernels reach on this device, as a
// reference for the pipeline's own rates (a standalone program, not part of
// the library).  Four kernels over 4 GiB, 16 bytes per lane, grid-stride
// loops: read only, write only, copy, and copy with one read written to three
// places (the 1:3 read:write mix of the row copy at the default workload).
// Then row gathers out[dst[i]] = table[src[i]] over 2 GiB of 256-B and 1-KiB
// rows of an 8 GiB table: random sources with sequential destinations, with
// random destinations (a permutation), and with random destinations plus a
// lone 4-B id store per row at its destination index, the access pattern of
// the row copy, which writes each row where its minibatch needs it.  Stores
// are non-temporal, as in the row copy.  Prints one JSON line per kernel:
// best and mean rate over 10 timed launches (row gathers: row bytes read and
// written only).  Last, lone 4-byte stores: 3.2 M of them into a 12.8 MB
// array (the column stores of the join at the default workload), consecutive,
// at a random permutation of the places, random inside one eighth of the array
// per XCD (workgroup w takes eighth w mod 8: workgroups are dealt to the XCDs
// in turn), and in runs of 10 consecutive places per lane (the sampler's
// pattern); and 4 M lone 4-byte loads at random places of a 1 GiB table (the
// sampler's neighbour reads), 8 independent loads per lane: best of 10
// launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <numeric>
#include <random>
#include <vector>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;
constexpr int kWave = 64;
constexpr int kGrid = 8192;
constexpr int kUnroll = 8;
constexpr int kReps = 10;

#define CHECK(x)                                                                            \
    do {                                                                                    \
        hipError_t e_ = (x);                                                                \
        if (e_ != hipSuccess) {                                                             \
            std::fprintf(stderr, "hbm_ceiling: %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            std::exit(1);                                                                   \
        }                                                                                   \
    } while (0)

// Read n units; the xor of everything goes to sink[0] only if it matches an
// arbitrary pattern (never, for the filled input), so the loads stay live.
__global__ __launch_bounds__(kBlock) void k_read(const u32x4* __restrict__ a, size_t n, u32x4* sink) {
    u32x4 acc = {0u, 0u, 0u, 0u};
    const size_t stride = (size_t)gridDim.x * kBlock * kUnroll;
    for (size_t b = (size_t)blockIdx.x * kBlock * kUnroll + threadIdx.x; b < n; b += stride) {
        u32x4 x[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; k++) {
            const size_t i = b + (size_t)k * kBlock;
            x[k] = i < n ? a[i] : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int k = 0; k < kUnroll; k++) acc ^= x[k];
    }
    if (acc.x == 0x9e3779b9u && acc.y == 0x7f4a7c15u && acc.z == 0x85ebca6bu) sink[0] = acc;
}

__global__ __launch_bounds__(kBlock) void k_write(u32x4* __restrict__ o, size_t n) {
    const size_t stride = (size_t)gridDim.x * kBlock * kUnroll;
    for (size_t b = (size_t)blockIdx.x * kBlock * kUnroll + threadIdx.x; b < n; b += stride) {
#pragma unroll
        for (int k = 0; k < kUnroll; k++) {
            const size_t i = b + (size_t)k * kBlock;
            if (i < n) __builtin_nontemporal_store(u32x4{(unsigned)i, 1u, 2u, 3u}, o + i);
        }
    }
}

// Copy a[0, n) to `copies` consecutive output ranges of n units each.
__global__ __launch_bounds__(kBlock) void k_copy(const u32x4* __restrict__ a, u32x4* __restrict__ o, size_t n,
                                                 int copies) {
    const size_t stride = (size_t)gridDim.x * kBlock * kUnroll;
    for (size_t b = (size_t)blockIdx.x * kBlock * kUnroll + threadIdx.x; b < n; b += stride) {
        u32x4 x[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; k++) {
            const size_t i = b + (size_t)k * kBlock;
            if (i < n) x[k] = a[i];
        }
        for (int r = 0; r < copies; r++) {
#pragma unroll
            for (int k = 0; k < kUnroll; k++) {
                const size_t i = b + (size_t)k * kBlock;
                if (i < n) __builtin_nontemporal_store(x[k], o + (size_t)r * n + i);
            }
        }
    }
}

// One row of RU 16-byte units per group of RU lanes, U rows in flight per
// group; entries [0, n) of src / dst.
template <int RU, int U, bool IDS>
__global__ __launch_bounds__(kBlock) void k_rows(const u32x4* __restrict__ table, u32x4* __restrict__ out,
                                                 const int* __restrict__ src, const int* __restrict__ dst,
                                                 int* __restrict__ ids, long n) {
    constexpr int GPW = kWave / RU;                 // row groups per wave
    const int lane = threadIdx.x % kWave, g = lane / RU, li = lane % RU;
    const long wave = (long)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    const long nw = (long)gridDim.x * (kBlock / kWave);
    for (long r0 = (wave * GPW + g) * U; r0 < n; r0 += nw * GPW * U) {
        int s[U], d[U];
        u32x4 x[U];
#pragma unroll
        for (int k = 0; k < U; k++) {
            s[k] = r0 + k < n ? src[r0 + k] : 0;
            d[k] = r0 + k < n ? dst[r0 + k] : 0;
        }
#pragma unroll
        for (int k = 0; k < U; k++)
            if (r0 + k < n) x[k] = table[(long)s[k] * RU + li];
#pragma unroll
        for (int k = 0; k < U; k++) {
            if (r0 + k < n) {
                __builtin_nontemporal_store(x[k], out + (long)d[k] * RU + li);
                if (IDS && li == 0) ids[d[k]] = s[k];
            }
        }
    }
}

// Lone 4-byte stores.  mode 0: out[i]; 1: out[perm[i]]; 2: workgroup w
// stores the permutation of eighth c = w mod 8 (perm8 holds, at [c m, (c+1) m),
// a permutation of those places); 3: runs of R consecutive places per lane
// (start[q] for q < n / R).
template <int MODE, int R>
__global__ __launch_bounds__(kBlock) void k_stores(int* __restrict__ out, const int* __restrict__ perm, long n) {
    if (MODE == 2) {
        const long m = n / 8, parts = gridDim.x / 8, part = blockIdx.x / 8;
        const long c = blockIdx.x % 8;
        for (long i = part * kBlock + threadIdx.x; i < m; i += parts * kBlock) out[perm[c * m + i]] = (int)i;
    } else if (MODE == 3) {
        for (long q = (long)blockIdx.x * kBlock + threadIdx.x; q < n / R; q += (long)gridDim.x * kBlock) {
            const int s0 = perm[q];
#pragma unroll
            for (int r = 0; r < R; r++) out[s0 + r] = r;
        }
    } else {
        for (long i = (long)blockIdx.x * kBlock + threadIdx.x; i < n; i += (long)gridDim.x * kBlock)
            out[MODE == 1 ? perm[i] : i] = (int)i;
    }
}

// Lone 4-byte loads: 8 per lane, all issued before any is used; the xor of
// everything goes to sink[0] only if it matches an arbitrary pattern.
__global__ __launch_bounds__(kBlock) void k_loads(const int* __restrict__ tab, const unsigned* __restrict__ idx,
                                                  long n, int* sink) {
    constexpr int R = 8;
    for (long i = ((long)blockIdx.x * kBlock + threadIdx.x) * R; i < n; i += (long)gridDim.x * kBlock * R) {
        int v[R];
#pragma unroll
        for (int r = 0; r < R; r++) v[r] = tab[idx[i + r]];
        int acc = 0;
#pragma unroll
        for (int r = 0; r < R; r++) acc ^= v[r];
        if (acc == 0x2545f491) sink[0] = acc;
    }
}

}  // namespace

int main() {
    const size_t bytes = (size_t)4 << 30, n = bytes / sizeof(u32x4);
    u32x4 *a = nullptr, *o = nullptr, *sink = nullptr;
    CHECK(hipMalloc(&a, bytes));
    CHECK(hipMalloc(&o, 3 * bytes));
    CHECK(hipMalloc(&sink, sizeof(u32x4)));
    CHECK(hipMemset(a, 1, bytes));
    CHECK(hipMemset(o, 0, 3 * bytes));
    CHECK(hipDeviceSynchronize());
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    auto timed = [&](const char* name, double moved, int grid, auto launch) {
        launch();
        CHECK(hipGetLastError());
        CHECK(hipDeviceSynchronize());
        float best = 1e30f, total = 0.f;
        for (int r = 0; r < kReps; r++) {
            CHECK(hipEventRecord(e0, 0));
            launch();
            CHECK(hipEventRecord(e1, 0));
            CHECK(hipEventSynchronize(e1));
            float ms = 0.f;
            CHECK(hipEventElapsedTime(&ms, e0, e1));
            best = ms < best ? ms : best;
            total += ms;
        }
        std::printf("{\"kernel\": \"%s\", \"bytes\": %.0f, \"best_ms\": %.4f, \"best_GBps\": %.1f, "
                    "\"mean_GBps\": %.1f, \"grid\": %d, \"launches\": %d}\n",
                    name, moved, best, moved / best / 1e6, moved / (total / kReps) / 1e6, grid, kReps);
        std::fflush(stdout);
    };
    const double B = (double)bytes;
    timed("read", B, kGrid, [&] { hipLaunchKernelGGL(k_read, dim3(kGrid), dim3(kBlock), 0, 0, a, n, sink); });
    timed("write", B, kGrid, [&] { hipLaunchKernelGGL(k_write, dim3(kGrid), dim3(kBlock), 0, 0, o, n); });
    timed("copy", 2 * B, kGrid, [&] { hipLaunchKernelGGL(k_copy, dim3(kGrid), dim3(kBlock), 0, 0, a, o, n, 1); });
    timed("copy 1:3", 4 * B, kGrid, [&] { hipLaunchKernelGGL(k_copy, dim3(kGrid), dim3(kBlock), 0, 0, a, o, n, 3); });
    // row gathers: rows of an 8 GiB table of their own, 2 GiB of them written
    // into the first 2 GiB of o
    {
        const size_t tbytes = (size_t)8 << 30, obytes = (size_t)2 << 30;
        u32x4* table = nullptr;
        CHECK(hipMalloc(&table, tbytes));
        CHECK(hipMemset(table, 3, tbytes));
        u32x4* rows_out = o;                            // 12 GiB buffer: rows use the first 2 GiB
        int *src = nullptr, *seq = nullptr, *perm = nullptr, *ids = nullptr;
        const long nmax = (long)(obytes / 256);
        CHECK(hipMalloc(&src, nmax * sizeof(int)));
        CHECK(hipMalloc(&seq, nmax * sizeof(int)));
        CHECK(hipMalloc(&perm, nmax * sizeof(int)));
        CHECK(hipMalloc(&ids, nmax * sizeof(int)));
        std::vector<int> h((size_t)nmax);
        for (int rb : {256, 1024}) {
            const long n = (long)(obytes / rb), nt = (long)(tbytes / rb);
            std::mt19937_64 rng(rb);
            for (long i = 0; i < n; i++) h[i] = (int)(rng() % (unsigned long long)nt);
            CHECK(hipMemcpy(src, h.data(), n * sizeof(int), hipMemcpyHostToDevice));
            std::iota(h.begin(), h.begin() + n, 0);
            CHECK(hipMemcpy(seq, h.data(), n * sizeof(int), hipMemcpyHostToDevice));
            std::shuffle(h.begin(), h.begin() + n, rng);
            CHECK(hipMemcpy(perm, h.data(), n * sizeof(int), hipMemcpyHostToDevice));
            const double moved = 2.0 * (double)obytes;
            char name[96];
            auto launch = [&](const int* dst, bool with_ids) {
                if (rb == 256) {
                    if (with_ids)
                        hipLaunchKernelGGL((k_rows<16, 4, true>), dim3(kGrid * 8), dim3(kBlock), 0, 0, table,
                                           rows_out, src, dst, ids, n);
                    else
                        hipLaunchKernelGGL((k_rows<16, 4, false>), dim3(kGrid * 8), dim3(kBlock), 0, 0, table,
                                           rows_out, src, dst, ids, n);
                } else {
                    if (with_ids)
                        hipLaunchKernelGGL((k_rows<64, 4, true>), dim3(kGrid * 8), dim3(kBlock), 0, 0, table,
                                           rows_out, src, dst, ids, n);
                    else
                        hipLaunchKernelGGL((k_rows<64, 4, false>), dim3(kGrid * 8), dim3(kBlock), 0, 0, table,
                                           rows_out, src, dst, ids, n);
                }
            };
            std::snprintf(name, sizeof(name), "rows %d B: random sources, sequential destinations", rb);
            timed(name, moved, kGrid * 8, [&] { launch(seq, false); });
            std::snprintf(name, sizeof(name), "rows %d B: random sources, random destinations", rb);
            timed(name, moved, kGrid * 8, [&] { launch(perm, false); });
            std::snprintf(name, sizeof(name), "rows %d B: random sources and destinations, 4-B id per row", rb);
            timed(name, moved, kGrid * 8, [&] { launch(perm, true); });
        }
        CHECK(hipFree(table));
        CHECK(hipFree(src));
        CHECK(hipFree(seq));
        CHECK(hipFree(perm));
        CHECK(hipFree(ids));
    }
    // lone 4-byte stores
    {
        const long n = 3200000, m = n / 8;      // n is a multiple of 80
        int *out = nullptr, *perm = nullptr, *perm8 = nullptr, *starts = nullptr;
        CHECK(hipMalloc(&out, n * sizeof(int)));
        CHECK(hipMalloc(&perm, n * sizeof(int)));
        CHECK(hipMalloc(&perm8, n * sizeof(int)));
        CHECK(hipMalloc(&starts, n / 10 * sizeof(int)));
        std::vector<int> h((size_t)n);
        std::mt19937_64 rng(7);
        std::iota(h.begin(), h.end(), 0);
        std::shuffle(h.begin(), h.end(), rng);
        CHECK(hipMemcpy(perm, h.data(), n * sizeof(int), hipMemcpyHostToDevice));
        std::iota(h.begin(), h.end(), 0);
        for (int c = 0; c < 8; c++) std::shuffle(h.begin() + c * m, h.begin() + (c + 1) * m, rng);
        CHECK(hipMemcpy(perm8, h.data(), n * sizeof(int), hipMemcpyHostToDevice));
        for (long q = 0; q < n / 10; q++) h[q] = (int)(q * 10);
        std::shuffle(h.begin(), h.begin() + n / 10, rng);
        CHECK(hipMemcpy(starts, h.data(), n / 10 * sizeof(int), hipMemcpyHostToDevice));
        const double moved = 4.0 * (double)n;
        const int g = 2048;
        timed("4-B stores: consecutive", moved, g,
              [&] { hipLaunchKernelGGL((k_stores<0, 1>), dim3(g), dim3(kBlock), 0, 0, out, perm, n); });
        timed("4-B stores: random permutation", moved, g,
              [&] { hipLaunchKernelGGL((k_stores<1, 1>), dim3(g), dim3(kBlock), 0, 0, out, perm, n); });
        timed("4-B stores: random inside one eighth per XCD", moved, g,
              [&] { hipLaunchKernelGGL((k_stores<2, 1>), dim3(g), dim3(kBlock), 0, 0, out, perm8, n); });
        timed("4-B stores: runs of 10 per lane", moved, g,
              [&] { hipLaunchKernelGGL((k_stores<3, 10>), dim3(g), dim3(kBlock), 0, 0, out, starts, n); });
        CHECK(hipFree(out));
        CHECK(hipFree(perm));
        CHECK(hipFree(perm8));
        CHECK(hipFree(starts));
    }
    // lone 4-byte loads
    {
        const long tn = 1L << 28, n = 1L << 22;   // a 1 GiB table; n is a multiple of 8
        int* tab = nullptr;
        unsigned* idx = nullptr;
        CHECK(hipMalloc(&tab, tn * sizeof(int)));
        CHECK(hipMalloc(&idx, n * sizeof(unsigned)));
        CHECK(hipMemset(tab, 1, tn * sizeof(int)));
        std::vector<unsigned> h((size_t)n);
        std::mt19937_64 rng(11);
        for (long i = 0; i < n; i++) h[i] = (unsigned)(rng() % (unsigned long long)tn);
        CHECK(hipMemcpy(idx, h.data(), n * sizeof(unsigned), hipMemcpyHostToDevice));
        const int g = 4096;
        timed("4-B loads: random places of a 1 GiB table", 4.0 * (double)n, g,
              [&] { hipLaunchKernelGGL(k_loads, dim3(g), dim3(kBlock), 0, 0, tab, idx, n, (int*)sink); });
        CHECK(hipFree(tab));
        CHECK(hipFree(idx));
    }
    CHECK(hipFree(a));
    CHECK(hipFree(o));
    CHECK(hipFree(sink));
    return 0;
}
