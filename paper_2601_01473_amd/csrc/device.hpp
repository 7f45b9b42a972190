// Device-side building blocks shared by the gfx950 kernels: wave64 primitives,
// workgroup scans, the counter-based RNG and Floyd's subset sampler.  Everything here is written for 64-lane
// wavefronts and 256-thread workgroups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace agnes {

constexpr int kWave = 64;
constexpr int kBlock = 256;                 // threads per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kXcds = 8;                    // accelerator dies of the chip; workgroups are dealt to them in turn

__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / kWave; }
__device__ __forceinline__ uint64_t lanemask_lt() {
    return (lane_id() == 0) ? 0ull : (~0ull >> (64 - lane_id()));
}

// Read lane `src` of a 64-bit value (all lanes must participate).
__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = (uint32_t)__shfl((int)lo, src, kWave);
    hi = (uint32_t)__shfl((int)hi, src, kWave);
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum over the 64 lanes of a wave.
template <typename T>
__device__ __forceinline__ T wave_inclusive_scan(T v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        T o = __shfl_up(v, d, kWave);
        if (lane_id() >= d) v += o;
    }
    return v;
}

// Exclusive prefix sum over a 256-thread workgroup; also returns the total.
// `lds` must hold kWavesPerBlock elements; the call contains barriers.
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T* lds, T& total) {
    T inc = wave_inclusive_scan(v);
    if (lane_id() == kWave - 1) lds[wave_id()] = inc;
    __syncthreads();
    T base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; w++) {
        T x = lds[w];
        if (w < wave_id()) base += x;
        tot += x;
    }
    __syncthreads();
    total = tot;
    return base + inc - v;
}

// Index j with off[j] <= x < off[j+1] for a nondecreasing off[0..n] (x < off[n]).
template <typename T>
__device__ __forceinline__ int upper_segment(const T* off, int n, T x) {
    int lo = 0, hi = n;   // invariant: off[lo] <= x < off[hi]
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (off[mid] <= x) lo = mid; else hi = mid;
    }
    return lo;
}

// upper_segment for Q values at once: the halving steps depend on n only, so
// the Q searches advance together and their LDS reads overlap.  Every x[q] <
// off[n].
template <int Q, typename T>
__device__ __forceinline__ void upper_segments(const T* off, int n, const T (&x)[Q], int (&out)[Q]) {
#pragma unroll
    for (int q = 0; q < Q; q++) out[q] = 0;
    int len = n;   // invariant: off[out] <= x < off[out + len]
    while (len > 1) {
        const int half = len >> 1;
#pragma unroll
        for (int q = 0; q < Q; q++) out[q] = off[out[q] + half] <= x[q] ? out[q] + half : out[q];
        len -= half;
    }
}

// The same search by a group of P lanes (P divides 64; lanes [g*P, (g+1)*P)
// form group g and the groups of a wave search independently): log_P(n) rounds
// of P probes.  All lanes of a group must call it together.
template <int P, typename Pred>
__device__ __forceinline__ int64_t group_partition_point(int64_t lo, int64_t hi, Pred before) {
    const int gl = lane_id() % P;
    const uint64_t gmask = (P == kWave) ? ~0ull : (((1ull << P) - 1) << (lane_id() - gl));
    while (lo < hi) {
        const int64_t n = hi - lo;
        const int64_t step = (n + P - 1) / P;
        const int64_t p = lo + (int64_t)gl * step;
        const bool probe = p < hi;
        const int c = __popcll(__ballot(probe && before(p)) & gmask);
        if (c == 0) return lo;
        const int probes = (int)((n + step - 1) / step);
        const int64_t nhi = c < probes ? lo + (int64_t)c * step : hi;
        lo = lo + (int64_t)(c - 1) * step + 1;
        hi = nhi;
    }
    return lo;
}

// First index in [lo, hi) where before() is false, for a predicate that is true
// on a prefix of the range, searched by one wave: every round the 64 lanes test
// 64 evenly spaced indices, which narrows the range by a factor of ~64, so a
// search over n entries costs about log64(n) memory round trips.  All lanes of
// the wave must call it and all get the answer.
template <typename Pred>
__device__ __forceinline__ int64_t wave_partition_point(int64_t lo, int64_t hi, Pred before) {
    const int lane = lane_id();
    while (lo < hi) {
        const int64_t n = hi - lo;
        const int64_t step = (n + kWave - 1) / kWave;
        const int64_t p = lo + (int64_t)lane * step;
        const bool probe = p < hi;
        const int c = __popcll(__ballot(probe && before(p)));
        if (c == 0) return lo;
        const int probes = (int)((n + step - 1) / step);
        const int64_t nlo = lo + (int64_t)(c - 1) * step + 1;
        const int64_t nhi = c < probes ? lo + (int64_t)c * step : hi;
        lo = nlo;
        hi = nhi;
    }
    return lo;
}

// ----------------------------------------------------------------- device-wide scan layout

// A scan over n elements (n read on the device) is split into G ranges of
// whole tiles, one per workgroup: a reduce pass writes each range's sum, a
// final pass adds the sums before its range and scans it.
constexpr int kScanGroups = 1024;   // partial sums per scan
constexpr int kScanItems = 4;       // consecutive elements per thread per tile
constexpr int kScanTile = kBlock * kScanItems;

__device__ __forceinline__ void scan_range(int64_t n, int G, int g, int64_t& lo, int64_t& hi) {
    int64_t chunk = (n + G - 1) / G;
    chunk = (chunk + kScanTile - 1) / kScanTile * kScanTile;
    lo = (int64_t)g * chunk;
    if (lo > n) lo = n;
    hi = lo + chunk;
    if (hi > n) hi = n;
}

// ----------------------------------------------------------------- RNG

// Philox4x64 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC 2011): two 64x64->128
// multiplies per round with the published multipliers, key bumped by the
// published Weyl increments between rounds.
struct Words4 { uint64_t w[4]; };

// Full 128-bit product of a 64-bit constant and a 64-bit value from four
// 32 x 32 -> 64 multiply-adds (each partial sum fits in 64 bits).
__device__ __forceinline__ void mul64_wide(uint64_t a, uint64_t b, uint64_t& hi, uint64_t& lo) {
    const uint64_t al = (uint32_t)a, ah = a >> 32, bl = (uint32_t)b, bh = b >> 32;
    const uint64_t t0 = al * bl;
    const uint64_t t1 = al * bh + (t0 >> 32);
    const uint64_t t2 = ah * bl + (uint32_t)t1;
    hi = ah * bh + (t1 >> 32) + (t2 >> 32);
    lo = (t2 << 32) | (uint32_t)t0;
}

__device__ __forceinline__ Words4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        uint64_t hi0, lo0, hi1, lo1;
        mul64_wide(M0, c0, hi0, lo0);
        mul64_wide(M1, c2, hi1, lo1);
        uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
        k0 += W0; k1 += W1;
    }
    Words4 o;
    o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
    return o;
}

// floor(w * n / 2^64): an integer in [0, n).
__device__ __forceinline__ uint64_t draw_below(uint64_t w, uint64_t n) { return __umul64hi(w, n); }

// ----------------------------------------------------------------- Floyd

// Floyd's algorithm for k of deg positions of node v (k < deg): draw i
// (i = 0..k-1) picks d in [0, t], t = deg - k + i, and keeps t when d was
// already chosen.  Word i comes from Philox(counter (i>>2, v, m, l), key
// (seed, 0)), lane i & 3.  pos[0..k) receives the positions in draw order; MAXK >= k.
template <int MAXK>
__device__ __forceinline__ void floyd_positions(uint64_t deg, int k, uint64_t seed, uint64_t v, uint64_t m,
                                                uint64_t l, uint32_t (&pos)[MAXK]) {
    Words4 words;
#pragma unroll
    for (int i = 0; i < MAXK; i++) {
        if (i < k) {
            if ((i & 3) == 0) words = philox4x64_10((uint64_t)(i >> 2), v, m, l, seed, 0);
            uint64_t t = deg - (uint64_t)k + (uint64_t)i;
            uint32_t d = (uint32_t)draw_below(words.w[i & 3], t + 1);
            bool seen = false;
#pragma unroll
            for (int s = 0; s < MAXK; s++)
                if (s < i) seen |= (pos[s] == d);
            pos[i] = seen ? (uint32_t)t : d;
        }
    }
}

// Neighbours at positions pos[0..k) of row adj written to out[0..k) in
// ascending position order (the slot of a position is its rank).  Every load is
// issued before the first store, so a request waits for one memory round trip.
template <int MAXK>
__device__ __forceinline__ void write_ranked(const uint32_t (&pos)[MAXK], int k, const int32_t* adj,
                                             int32_t* out) {
    int32_t val[MAXK];
#pragma unroll
    for (int a = 0; a < MAXK; a++)
        if (a < k) val[a] = adj[pos[a]];
#pragma unroll
    for (int a = 0; a < MAXK; a++) {
        if (a < k) {
            int rank = 0;
#pragma unroll
            for (int b = 0; b < MAXK; b++)
                if (b < k) rank += (pos[b] < pos[a]) ? 1 : 0;
            out[rank] = val[a];
        }
    }
}

// Any k: the positions are staged in out[0..k) itself, sorted, then replaced by
// the neighbours eight at a time.
__device__ __forceinline__ void floyd_sample_mem(uint64_t deg, int k, uint64_t seed, uint64_t v,
                                                 uint64_t m, uint64_t l, const int32_t* adj,
                                                 int32_t* out) {
    Words4 words;
    for (int i = 0; i < k; i++) {
        if ((i & 3) == 0) words = philox4x64_10((uint64_t)(i >> 2), v, m, l, seed, 0);
        uint64_t t = deg - (uint64_t)k + (uint64_t)i;
        int32_t d = (int32_t)draw_below(words.w[i & 3], t + 1);
        bool seen = false;
        for (int s = 0; s < i; s++) seen |= (out[s] == d);
        out[i] = seen ? (int32_t)t : d;
    }
    for (int i = 1; i < k; i++) {            // insertion sort of the positions
        int32_t x = out[i];
        int s = i - 1;
        while (s >= 0 && out[s] > x) { out[s + 1] = out[s]; s--; }
        out[s + 1] = x;
    }
    for (int i0 = 0; i0 < k; i0 += 8) {
        int32_t p[8], x[8];
#pragma unroll
        for (int t = 0; t < 8; t++)
            if (i0 + t < k) p[t] = out[i0 + t];
#pragma unroll
        for (int t = 0; t < 8; t++)
            if (i0 + t < k) x[t] = adj[p[t]];
#pragma unroll
        for (int t = 0; t < 8; t++)
            if (i0 + t < k) out[i0 + t] = x[t];
    }
}

// A whole row (k == deg), eight neighbours at a time.
__device__ __forceinline__ void copy_row(const int32_t* adj, int k, int32_t* out) {
    for (int i0 = 0; i0 < k; i0 += 8) {
        int32_t x[8];
#pragma unroll
        for (int t = 0; t < 8; t++)
            if (i0 + t < k) x[t] = adj[i0 + t];
#pragma unroll
        for (int t = 0; t < 8; t++)
            if (i0 + t < k) out[i0 + t] = x[t];
    }
}

}  // namespace agnes
