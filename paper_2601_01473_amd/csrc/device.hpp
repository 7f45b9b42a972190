// Device-side building blocks shared by the gfx950 kernels: wave64 primitives,
// workgroup scans, the counter-based RNG, Floyd's subset sampler and the
// (minibatch, node) hash table.  Everything here is written for 64-lane
// wavefronts and 256-thread workgroups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace agnes {

constexpr int kWave = 64;
constexpr int kBlock = 256;                 // threads per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;

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

// Wave-aggregated atomicAdd of 1 per active lane on counters[key]: lanes sharing
// a key are combined into one atomic.  Returns, per lane, the counter value its
// own increment corresponds to (base + rank among same-key lanes, in lane order)
// and sets `first` on the one lane (the group's lowest) whose group found the
// counter at zero.
__device__ __forceinline__ int64_t wave_aggregated_increment(int64_t* counters, int64_t key,
                                                             bool active, bool& first) {
    uint64_t todo = __ballot(active);
    int64_t result = 0;
    first = false;
    while (todo) {
        int leader = __ffsll((unsigned long long)todo) - 1;
        int64_t k = (int64_t)shfl64((uint64_t)key, leader);
        uint64_t peers = __ballot(active && key == k) & todo;
        int64_t base = 0;
        if (lane_id() == leader)
            base = atomicAdd((unsigned long long*)&counters[k], (unsigned long long)__popcll(peers));
        base = (int64_t)shfl64((uint64_t)base, leader);
        if (peers & (1ull << lane_id())) {
            result = base + __popcll(peers & lanemask_lt());
            first = (base == 0) && (lane_id() == leader);
        }
        todo &= ~peers;
    }
    return result;
}

// Wave-aggregated atomicAdd of 1 per active lane on a single counter.
__device__ __forceinline__ int64_t wave_append(int64_t* counter, bool active) {
    uint64_t m = __ballot(active);
    if (m == 0) return -1;
    int leader = __ffsll((unsigned long long)m) - 1;
    int64_t base = 0;
    if (lane_id() == leader) base = atomicAdd((unsigned long long*)counter, (unsigned long long)__popcll(m));
    base = (int64_t)shfl64((uint64_t)base, leader);
    return active ? base + __popcll(m & lanemask_lt()) : -1;
}

// ----------------------------------------------------------------- RNG

// Philox4x64 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC 2011): two 64x64->128
// multiplies per round with the published multipliers, key bumped by the
// published Weyl increments between rounds.
struct Words4 { uint64_t w[4]; };

__device__ __forceinline__ Words4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
        uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
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

// Sample k of deg positions of node v (k < deg) and write the neighbours at those
// positions, in ascending position order, to out[0..k).  Floyd's algorithm: draw
// i (i = 0..k-1) picks d in [0, t], t = deg - k + i, and keeps t when d was
// already chosen.  Word i comes from Philox(counter (i>>2, v, m, l), key (seed, 0)),
// lane i & 3.  Positions live in registers; MAXK >= k.
template <int MAXK>
__device__ __forceinline__ void floyd_sample_regs(uint64_t deg, int k, uint64_t seed, uint64_t v,
                                                  uint64_t m, uint64_t l, const int32_t* adj,
                                                  int32_t* out) {
    uint32_t pos[MAXK];
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
    // the output slot of a position is its rank among the chosen positions
#pragma unroll
    for (int a = 0; a < MAXK; a++) {
        if (a < k) {
            int rank = 0;
#pragma unroll
            for (int b = 0; b < MAXK; b++)
                if (b < k) rank += (pos[b] < pos[a]) ? 1 : 0;
            out[rank] = adj[pos[a]];
        }
    }
}

// Same sampler for any k: the positions are staged in out[0..k) itself.
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
    for (int i = 0; i < k; i++) out[i] = adj[out[i]];
}

// ----------------------------------------------------------------- hash table

// Open addressing with linear probing over 64-bit words.  A word holds
// (generation << kKeyBits) | key; words of another generation count as empty, so
// the table is reused across hyperbatches without being cleared.  Keys are
// (minibatch << node_bits) | node.
constexpr int kKeyBits = 44;
constexpr uint64_t kKeyMask = (1ull << kKeyBits) - 1;

__device__ __forceinline__ uint64_t ht_hash(uint64_t key, int log2cap) {
    return (key * 0x9E3779B97F4A7C15ull) >> (64 - log2cap);
}

// Insert (or find) `key`; returns the slot and whether this call inserted it.
// Terminates because the table is sized to at least twice the keys of a
// hyperbatch and a word, once it holds a current-generation key, never changes.
__device__ __forceinline__ uint32_t ht_insert(unsigned long long* words, int log2cap, uint64_t gen,
                                              uint64_t key, bool& inserted) {
    const uint64_t mask = (1ull << log2cap) - 1;
    const unsigned long long tagged = (gen << kKeyBits) | key;
    uint64_t slot = ht_hash(key, log2cap);
    for (;;) {
        unsigned long long cur = __hip_atomic_load(&words[slot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (;;) {
            if (cur == tagged) { inserted = false; return (uint32_t)slot; }
            if ((cur >> kKeyBits) == gen) break;                 // another live key
            unsigned long long prev = atomicCAS(&words[slot], cur, tagged);
            if (prev == cur) { inserted = true; return (uint32_t)slot; }
            cur = prev;
        }
        slot = (slot + 1) & mask;
    }
}

}  // namespace agnes
