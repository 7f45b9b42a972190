// HBM ceiling probe: what plain streaming kernels reach on this device, as a
// reference for the pipeline's own rates (a standalone program, not part of
// the library).  Four kernels over 4 GiB, 16 bytes per lane, grid-stride
// loops: read only, write only, copy, and copy with one read written to three
// places (the 1:3 read:write mix of the row copy at the default workload).
// Stores are non-temporal, as in the row copy.  Prints one JSON line per
// kernel: best and mean rate over 10 timed launches.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;
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
    auto timed = [&](const char* name, double moved, auto launch) {
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
                    name, moved, best, moved / best / 1e6, moved / (total / kReps) / 1e6, kGrid, kReps);
        std::fflush(stdout);
    };
    const double B = (double)bytes;
    timed("read", B, [&] { hipLaunchKernelGGL(k_read, dim3(kGrid), dim3(kBlock), 0, 0, a, n, sink); });
    timed("write", B, [&] { hipLaunchKernelGGL(k_write, dim3(kGrid), dim3(kBlock), 0, 0, o, n); });
    timed("copy", 2 * B, [&] { hipLaunchKernelGGL(k_copy, dim3(kGrid), dim3(kBlock), 0, 0, a, o, n, 1); });
    timed("copy 1:3", 4 * B, [&] { hipLaunchKernelGGL(k_copy, dim3(kGrid), dim3(kBlock), 0, 0, a, o, n, 3); });
    CHECK(hipFree(a));
    CHECK(hipFree(o));
    CHECK(hipFree(sink));
    return 0;
}
